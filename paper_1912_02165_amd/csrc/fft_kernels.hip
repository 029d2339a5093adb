// FFT-tile fused 3x3 convolution for gfx950 (the FFT transform of Sec. 2.1 and
// Sec. 4 with the fusion of Sec. 3): 16x16 input tiles overlapping by 2 give
// 14x14 output tiles; a tile's spectrum is conjugate symmetric, so only the
// 16 x 9 frequencies with column index q <= 8 are kept (Sec. 2.1).
//
// Per frequency f = p*9 + q the contraction over input channels is complex:
//     Z[f][k][t] = sum_c D[f][c][t] * conj(Wp[f][k][c])
// (the convolution theorem for the cross-correlation of Eq. 1; circular on the
// 16x16 tile, equal to the linear one on the 14x14 output tile).  With
// D = Dr + i Di and Wp = Wr + i Wi:
//     Re Z = sum Wr Dr + Wi Di,   Im Z = sum Wr Di + (-Wi) Dr,
// four real products per complex one, on v_mfma_f32_16x16x4_f32 with the
// output channels as rows (operand A, from the transformed kernels) and tiles as
// columns (operand B, from LDS).
//
// Work item = 16 tiles x 16 output channels, one workgroup of 8 waves each: the
// item's 16 x 16 x 144 complex sums (1.18 MB for 64 output channels) do not fit
// a compute unit, so an item holds one 16-channel block; wave w accumulates
// frequencies 18w .. 18w + 17 (36 accumulator tiles = 144 registers).  Per
// stage of 4 input channels: the 64 input tiles are loaded into LDS, transformed
// (16-point FFTs along rows, then along the 9 kept columns), and each wave runs
// its 72 products.  After the last stage the sums go back through LDS a quarter
// of the output channels at a time for the inverse transforms.
#include "wino_internal.h"

#include <hip/hip_runtime.h>

namespace wino {

typedef float fft_floatx4 __attribute__((ext_vector_type(4)));
typedef int fft_int32x4 __attribute__((ext_vector_type(4)));

// Raw buffer loads: an offset at or past the resource's size reads 0, which
// gives the zero padding of input windows without branches.  (Declared outside
// the anonymous namespace below: they name LLVM intrinsics, which have external
// linkage.)
__device__ float fft_buffer_load_f32(fft_int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.load.f32");
__device__ void fft_buffer_store_f32(float v, fft_int32x4 rsrc, unsigned voffset, unsigned soffset, int aux)
    __asm("llvm.amdgcn.raw.buffer.store.f32");

namespace {

typedef fft_floatx4 floatx4;
typedef fft_int32x4 int32x4;
__device__ __forceinline__ int32x4 fft_rsrc(const float *base, unsigned bytes) {
    const unsigned long long p = reinterpret_cast<unsigned long long>(base);
    int32x4 r;
    r[0] = (int)(unsigned)(p & 0xffffffffull);
    r[1] = (int)(unsigned)((p >> 32) & 0xffffull);  // stride 0
    r[2] = (int)bytes;                                 // range-checked size
    r[3] = 0x00020000;                                 // 32-bit data format
#pragma unroll
    for (int i = 0; i < 4; ++i) r[i] = __builtin_amdgcn_readfirstlane(r[i]);
    return r;
}
constexpr unsigned kFOutside = 0x80000000u;  // past every buffer (each is below 2^31 bytes)

constexpr int kFT = 16;             // tile edge
constexpr int kFM = 14;             // output tile edge
constexpr int kFQ = kFT / 2 + 1;    // kept spectrum columns
constexpr int kFF = kFT * kFQ;      // kept frequencies per tile (144)
constexpr int kFWaves = 8;
constexpr int kFPerWave = kFF / kFWaves;  // 18 frequencies per wave
static_assert(kFF % kFWaves == 0, "frequencies split evenly over the waves");

// cos(2 pi j / 16) and sin(2 pi j / 16): the 16th roots of unity, written out
// (cos(pi/8) = sqrt(2 + sqrt 2) / 2, cos(pi/4) = sqrt(2) / 2, cos(3 pi/8) =
// sqrt(2 - sqrt 2) / 2, rounded to float).
__host__ __device__ constexpr float cos16(int j) {
    switch (j & 15) {
        case 0: return 1.0f;
        case 1: case 15: return 0.923879532511286756f;
        case 2: case 14: return 0.707106781186547524f;
        case 3: case 13: return 0.382683432365089772f;
        case 4: case 12: return 0.0f;
        case 5: case 11: return -0.382683432365089772f;
        case 6: case 10: return -0.707106781186547524f;
        case 7: case 9: return -0.923879532511286756f;
        default: return -1.0f;
    }
}
__host__ __device__ constexpr float sin16(int j) { return cos16(j + 12); }  // sin x = cos(x - pi/2)

__host__ __device__ constexpr int bitrev4(int k) {
    return ((k & 1) << 3) | ((k & 2) << 1) | ((k & 4) >> 1) | ((k & 8) >> 3);
}

// In-place 16-point DFT X[a] = sum_b x[b] exp(S * 2 pi i a b / 16), S = -1
// (forward) or +1 (inverse, unscaled): radix-2 decimation in time.  The loops
// unroll completely, so every twiddle is a constant; the trivial ones (1 and
// +-i) are taken without multiplications.
template <int S>
__device__ __forceinline__ void dft16(float (&re)[16], float (&im)[16]) {
    float r[16], i[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        r[k] = re[bitrev4(k)];
        i[k] = im[bitrev4(k)];
    }
#pragma unroll
    for (int len = 2; len <= 16; len <<= 1) {
        const int half = len / 2;
#pragma unroll
        for (int s = 0; s < 16; s += len) {
#pragma unroll
            for (int j = 0; j < half; ++j) {
                const int tw = j * (16 / len);  // exp(S 2 pi i tw / 16)
                const int a = s + j, b = s + j + half;
                float xr, xi;
                if (tw == 0) {
                    xr = r[b];
                    xi = i[b];
                } else if (tw == 4) {  // multiply by S i
                    xr = -S * i[b];
                    xi = S * r[b];
                } else {
                    const float c = cos16(tw), sn = S * sin16(tw);
                    xr = r[b] * c - i[b] * sn;
                    xi = r[b] * sn + i[b] * c;
                }
                r[b] = r[a] - xr;
                i[b] = i[a] - xi;
                r[a] = r[a] + xr;
                i[a] = i[a] + xi;
            }
        }
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
        re[k] = r[k];
        im[k] = i[k];
    }
}

// Tile t of the layer: image n and tile row / column, as for the Winograd path
// with m = 14.
struct FTile {
    int n, ty, tx;
    bool ok;
};
__device__ __forceinline__ FTile fft_tile(const Geometry &g, int t) {
    FTile r;
    r.ok = t < g.ntiles;
    const int tt = r.ok ? t : 0;
    const int per = g.TH * g.TW;
    r.n = tt / per;
    const int rem = tt - r.n * per;
    r.ty = rem / g.TW;
    r.tx = rem - r.ty * g.TW;
    return r;
}

// Transformed kernels: wt[((cs * Kb + kb) * 144 + f) * 64 + lane] = {Re Wp,
// Im Wp, -Im Wp, 0} of output channel kb*16 + lane % 16 and input channel
// cs*4 + lane / 16 (the MFMA A-operand order), zero for padding channels.  One
// thread per (c, k), the spectrum summed from its definition (9 taps).
__global__ void __launch_bounds__(256) fft_weight_transform_kernel(const float *__restrict__ w,
                                                                    floatx4 *__restrict__ wt, Geometry g) {
    const int KP = g.Kb * 16;
    const long long total = (long long)g.Cs * 4 * KP;
    const long long idx = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (idx >= total) return;
    const int c = (int)(idx / KP), k = (int)(idx - (long long)c * KP);
    float tap[9];
    const bool ok = c < g.C && k < g.K;
#pragma unroll
    for (int e = 0; e < 9; ++e) tap[e] = ok ? w[((long long)k * g.C + c) * 9 + e] : 0.0f;
    const int lane = (c & 3) * 16 + (k & 15);
    floatx4 *dst = wt + ((long long)((c >> 2) * g.Kb + (k >> 4)) * kFF) * 64 + lane;
#pragma unroll
    for (int p = 0; p < kFT; ++p) {
#pragma unroll
        for (int q = 0; q < kFQ; ++q) {
            // Wp[p][q] = sum_{u,v} w[u][v] exp(-2 pi i (p u + q v) / 16)
            float re = 0.0f, im = 0.0f;
#pragma unroll
            for (int u = 0; u < 3; ++u)
#pragma unroll
                for (int v = 0; v < 3; ++v) {
                    const int a = p * u + q * v;
                    re += tap[u * 3 + v] * cos16(a);
                    im -= tap[u * 3 + v] * sin16(a);
                }
            dst[(p * kFQ + q) * 64] = floatx4{re, im, -im, 0.0f};
        }
    }
}

// Row transforms of two real rows at once: z = a + i b has spectrum Z, and
// A[q] = (Z[q] + conj Z[-q]) / 2, B[q] = (Z[q] - conj Z[-q]) / 2i.
__device__ __forceinline__ void unpack_real_pair(const float (&zr)[16], const float (&zi)[16], int q,
                                                 float &ar, float &ai, float &br, float &bi) {
    const int qc = (16 - q) & 15;
    ar = 0.5f * (zr[q] + zr[qc]);
    ai = 0.5f * (zi[q] - zi[qc]);
    br = 0.5f * (zi[q] + zi[qc]);
    bi = 0.5f * (zr[qc] - zr[q]);
}

__global__ void __launch_bounds__(512) fft_fused_kernel(const float *__restrict__ x,
                                                         const floatx4 *__restrict__ wt,
                                                         float *__restrict__ y, Geometry g) {
    // xin: the stage's 64 input tiles, element (tc, i, j) at tc * kXT + i * kXR + j,
    //      tc = channel-in-stage * 16 + tile (rows padded to 17 floats and tiles
    //      to 273, so that 64 lanes reading the same element of 64 tiles, or 16
    //      rows of one tile, fall in distinct banks)
    // spec: spectra [(f * 2 + part) * 64 + tc] (part 0 real, 1 imaginary), reused
    //       for the sums [(f * 2 + part) * 64 + lane] in the epilogue
    constexpr int kXR = 17, kXT = 273;
    __shared__ float xin[64 * kXT];
    __shared__ float spec[kFF * 2 * 64];
    // per tile of the item: x offset of its window's first element in channel 0
    // (may be negative: the window starts one row and column before the tile),
    // the rows (bits 0-15) and columns (bits 16-31) of the window inside the
    // image (0: no tile), the image, and the first output row and column
    __shared__ int tbase[16], tmask[16], tn[16], toy[16], tox[16];

    const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int tg = blockIdx.x / g.Kb, kb = blockIdx.x - tg * g.Kb;
    const long long HW = (long long)g.H * g.W;
    if (tid < 16) {
        const FTile ft = fft_tile(g, tg * 16 + tid);
        const int oy = ft.ty * kFM, ox = ft.tx * kFM;
        unsigned rows = 0, cols = 0;
        for (int e = 0; e < kFT; ++e) {
            if (oy - 1 + e >= 0 && oy - 1 + e < g.H) rows |= 1u << e;
            if (ox - 1 + e >= 0 && ox - 1 + e < g.W) cols |= 1u << e;
        }
        tbase[tid] = (int)((long long)ft.n * g.C * HW + (long long)(oy - 1) * g.W + (ox - 1));
        tmask[tid] = ft.ok ? (int)(rows | (cols << 16)) : 0;
        tn[tid] = ft.ok ? ft.n : -1;
        toy[tid] = oy;
        tox[tid] = ox;
    }

    floatx4 acc_re[kFPerWave], acc_im[kFPerWave];
#pragma unroll
    for (int j = 0; j < kFPerWave; ++j) {
        acc_re[j] = floatx4{0.f, 0.f, 0.f, 0.f};
        acc_im[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    }
    const floatx4 *wk = wt + (long long)kb * kFF * 64 + lane;  // + cs * Kb * 144 * 64
    __syncthreads();

    // Input element s (0..31) of this thread in a stage: tile-channel tc =
    // (tid >> 8) + 2 s (channel s >> 3, tile (tid >> 8) + 2 (s & 7)), window row
    // ei = (tid >> 4) & 15, column ej = tid & 15; 16 consecutive threads read one
    // window row.
    const int eh = tid >> 8, ei = (tid >> 4) & 15, ej = tid & 15;
    const int erel = ei * g.W + ej;
    const int32x4 xrs = fft_rsrc(x, (unsigned)((long long)g.N * g.C * HW * 4));
    const int32x4 yrs = fft_rsrc(y, (unsigned)((long long)g.N * g.K * HW * 4));
    float xr[32];
    auto load_stage = [&](int cs) {
#pragma unroll
        for (int s = 0; s < 32; ++s) {
            const int t = eh + 2 * (s & 7), ch = cs * 4 + (s >> 3);
            const unsigned msk = (unsigned)tmask[t];
            const bool in = ((msk >> ei) & (msk >> (16 + ej)) & 1u) && ch < g.C;
            // outside the window's valid part the offset gets the top bit (past the
            // buffer), without a branch around the load
            // (unsigned arithmetic: the unused offsets of padding channels may wrap)
            const unsigned el = (unsigned)tbase[t] + (unsigned)ch * (unsigned)HW + (unsigned)erel;
            const unsigned off = (el * 4u & ~kFOutside) | (in ? 0u : kFOutside);
            xr[s] = fft_buffer_load_f32(xrs, off, 0, 0);
        }
    };
    load_stage(0);

    for (int cs = 0; cs < g.Cs; ++cs) {
        // 1. the stage's input tiles (loaded during the previous stage's products)
#pragma unroll
        for (int s = 0; s < 32; ++s) xin[(eh + 2 * s) * kXT + ei * kXR + ej] = xr[s];
        __syncthreads();
        // kernel operands of the first frequencies, in flight during the transforms
        const floatx4 *ws = wk + (long long)cs * g.Kb * kFF * 64 + wave * kFPerWave * 64;
        constexpr int kCh = 3;  // frequencies per operand chunk
        floatx4 a0[kCh];
#pragma unroll
        for (int j = 0; j < kCh; ++j) a0[j] = ws[j * 64];
        // 2. along rows: rows i and i + 8 of tile-channel tc (= tid & 63, i = tid >> 6)
        //    as one complex transform; row i's 9 kept values go to spec at
        //    frequency i * 9 + q for now
        {
            const int tc = tid & 63, i = tid >> 6;
            float re[16], im[16];
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                re[j] = xin[tc * kXT + i * kXR + j];
                im[j] = xin[tc * kXT + (i + 8) * kXR + j];
            }
            dft16<-1>(re, im);
#pragma unroll
            for (int q = 0; q < kFQ; ++q) {
                float ar, ai, br, bi;
                unpack_real_pair(re, im, q, ar, ai, br, bi);
                spec[((i * kFQ + q) * 2 + 0) * 64 + tc] = ar;
                spec[((i * kFQ + q) * 2 + 1) * 64 + tc] = ai;
                spec[(((i + 8) * kFQ + q) * 2 + 0) * 64 + tc] = br;
                spec[(((i + 8) * kFQ + q) * 2 + 1) * 64 + tc] = bi;
            }
        }
        __syncthreads();
        // 3. along columns: 576 columns (tile-channel col & 63, column col >> 6),
        //    each transformed in place over its 16 rows
#pragma unroll 1
        for (int col = tid; col < 64 * kFQ; col += 512) {
            const int tc = col & 63, q = col >> 6;
            float re[16], im[16];
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                re[p] = spec[((p * kFQ + q) * 2 + 0) * 64 + tc];
                im[p] = spec[((p * kFQ + q) * 2 + 1) * 64 + tc];
            }
            dft16<-1>(re, im);
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                spec[((p * kFQ + q) * 2 + 0) * 64 + tc] = re[p];
                spec[((p * kFQ + q) * 2 + 1) * 64 + tc] = im[p];
            }
        }
        __syncthreads();
        // next stage's input tiles, in flight during the products
        if (cs + 1 < g.Cs) load_stage(cs + 1);
        // 4. products of the wave's frequencies: lane = channel-in-stage * 16 +
        //    tile reads operand B; its kernel operands {Wr, Wi, -Wi} come as one
        //    float4, the next chunk's loaded while one is multiplied
        floatx4 a1[kCh];
#pragma unroll
        for (int j0 = 0; j0 < kFPerWave; j0 += kCh) {
            if (j0 + kCh < kFPerWave) {
#pragma unroll
                for (int j = 0; j < kCh; ++j) a1[j] = ws[(j0 + kCh + j) * 64];
            }
#pragma unroll
            for (int j = 0; j < kCh; ++j) {
                const int f = wave * kFPerWave + j0 + j;
                const float br = spec[(f * 2 + 0) * 64 + lane], bi = spec[(f * 2 + 1) * 64 + lane];
                acc_re[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[j].x, br, acc_re[j0 + j], 0, 0, 0);
                acc_re[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[j].y, bi, acc_re[j0 + j], 0, 0, 0);
                acc_im[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[j].x, bi, acc_im[j0 + j], 0, 0, 0);
                acc_im[j0 + j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a0[j].z, br, acc_im[j0 + j], 0, 0, 0);
            }
#pragma unroll
            for (int j = 0; j < kCh; ++j) a0[j] = a1[j];
        }
        __syncthreads();  // xin and spec are rewritten by the next stage
    }

    // Epilogue, in four rounds v = 0..3: the sums of output channels
    // kb*16 + 4h + v (h = lane >> 4, accumulator element v) for tile lane & 15,
    // i.e. one sum per lane ("pair" = lane), pass through spec.
    constexpr float kScale = 1.0f / (kFT * kFT);
#pragma unroll
    for (int v = 0; v < 4; ++v) {
#pragma unroll
        for (int j = 0; j < kFPerWave; ++j) {
            const int f = wave * kFPerWave + j;
            spec[(f * 2 + 0) * 64 + lane] = acc_re[j][v];
            spec[(f * 2 + 1) * 64 + lane] = acc_im[j][v];
        }
        __syncthreads();
        // inverse along columns (pair col & 63, column col >> 6), in place; row p
        // of the result is output row p of the circular correlation
#pragma unroll 1
        for (int col = tid; col < 64 * kFQ; col += 512) {
            const int pr = col & 63, q = col >> 6;
            float re[16], im[16];
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                re[p] = spec[((p * kFQ + q) * 2 + 0) * 64 + pr];
                im[p] = spec[((p * kFQ + q) * 2 + 1) * 64 + pr];
            }
            dft16<1>(re, im);
#pragma unroll
            for (int p = 0; p < 16; ++p) {
                spec[((p * kFQ + q) * 2 + 0) * 64 + pr] = re[p];
                spec[((p * kFQ + q) * 2 + 1) * 64 + pr] = im[p];
            }
        }
        __syncthreads();
        // inverse along rows for output rows i and i + 7 (i < 7) of pair pr as one
        // complex transform: row i's spectrum (completed by conjugate symmetry,
        // imaginary parts at q = 0 and 8 dropped as for a real row) plus i times
        // row i + 7's gives row i in the real part, row i + 7 in the imaginary part
        if (tid < 64 * 7) {
            const int pr = tid & 63, i = tid >> 6;
            float re[16], im[16];
#pragma unroll
            for (int q = 0; q < kFQ; ++q) {
                const float ar = spec[((i * kFQ + q) * 2 + 0) * 64 + pr];
                const float ai = (q == 0 || q == 8) ? 0.0f : spec[((i * kFQ + q) * 2 + 1) * 64 + pr];
                const float br = spec[(((i + 7) * kFQ + q) * 2 + 0) * 64 + pr];
                const float bi = (q == 0 || q == 8) ? 0.0f : spec[(((i + 7) * kFQ + q) * 2 + 1) * 64 + pr];
                re[q] = ar - bi;
                im[q] = ai + br;
                if (q > 0 && q < 8) {  // column 16 - q: conj(A) + i conj(B)
                    re[16 - q] = ar + bi;
                    im[16 - q] = br - ai;
                }
            }
            dft16<1>(re, im);
            // stores outside the image (or of a missing tile or output channel)
            // get an offset past the buffer and are dropped
            const int t = pr & 15, k = kb * 16 + 4 * (pr >> 4) + v;
            const int n = tn[t], ox0 = tox[t];
            const bool ok = n >= 0 && k < g.K;
            // (unsigned arithmetic: offsets that are not used may wrap)
            const unsigned kbase = ((unsigned)(ok ? n : 0) * (unsigned)g.K + (unsigned)k) * (unsigned)HW;
#pragma unroll
            for (int half = 0; half < 2; ++half) {
                const int oy = toy[t] + i + 7 * half;
                const bool rok = ok && oy < g.H;
                const unsigned rowoff = (kbase + (unsigned)(oy * g.W + ox0)) * 4u;
#pragma unroll
                for (int j = 0; j < kFM; ++j) {
                    const unsigned off = (rok && ox0 + j < g.W) ? rowoff + 4u * j : kFOutside;
                    fft_buffer_store_f32((half ? im[j] : re[j]) * kScale, yrs, off, 0, 0);
                }
            }
        }
        __syncthreads();  // spec is rewritten by the next round
    }
}

}  // namespace

hipError_t launch_fft_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s) {
    const long long total = (long long)g.Cs * 4 * g.Kb * 16;
    const unsigned blocks = (unsigned)((total + 255) / 256);
    hipLaunchKernelGGL(fft_weight_transform_kernel, dim3(blocks), dim3(256), 0, s, w,
                       reinterpret_cast<floatx4 *>(wt), g);
    return hipGetLastError();
}

hipError_t launch_fft_fused(const Geometry &g, const float *x, const float *wt, float *y, hipStream_t s) {
    const long long items = (long long)((g.ntiles + 15) / 16) * g.Kb;
    hipLaunchKernelGGL(fft_fused_kernel, dim3((unsigned)items), dim3(512), 0, s, x,
                       reinterpret_cast<const floatx4 *>(wt), y, g);
    return hipGetLastError();
}

}  // namespace wino
