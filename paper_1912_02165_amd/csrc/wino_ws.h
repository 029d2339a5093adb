// The fused Winograd kernel (Sec. 4: a task of R tiles does input transform ->
// T^2 products against the hot kernel matrices -> output transform, its
// intermediates kept on chip), as a persistent, warp-specialised HIP kernel for
// gfx950.  wino_fused_inst.hip instantiates it once per built blocking
// (WINO_FUSED_BLOCKINGS in wino_internal.h), one object file each.
//
// A workgroup of 8 waves runs on one compute unit and processes a sequence of
// work items; an item (the paper's task) is R = 16*TB tiles x Kit output
// channels, Kit = 16 * KBW.
//
// Waves 4..7 are producers: per stage of CC = 256/R input channels each lane loads
// one (tile, channel) input tile, transforms it (B^T d B) and writes its T^2
// values to an LDS stage ring; loads run one or two stages ahead.
//
// Waves 0..3 are consumers on the matrix cores.  P = FS * CSP consumer waves share
// one 16-channel output block (so KBW = 4 / P blocks per item):
//   FS  frequency split: wave group G owns the transform-domain rows group_rows<G>
//       (needed for F(5) and F(6), whose T^2 frequencies would otherwise need 196
//       or 256 accumulator registers; for F(2) it halves an item's channels);
//   CSP channel-step split: wave part H multiplies channel steps H*SW .. H*SW+SW-1
//       of every stage (SW = SS / CSP).
// Each wave inverse-transforms its own partial sums (the output transform is
// linear: A^T (sum of parts) A = sum of A^T part A) and the P partial output tiles
// of a block are added in a fixed order through LDS slots.  The kernel operands
// of the next channel step are loaded while the current step runs.
//
// Two waves per SIMD (a producer and a consumer) let the producers' loads and
// vector work fill the gaps between the consumers' products.  Stage buffers are
// handed over through fill/drain counters in LDS instead of workgroup barriers.
//
// LDS layout of one stage buffer, in float4 units: [F4][CC][R] with the four
// frequencies 4*f4 .. 4*f4+3 of (channel, tile) in one float4, so that a wave's
// matrix-core B operand for four frequencies is one contiguous 1 KB read.
#pragma once

#include "wino_device.h"

namespace wino {

// Transform-domain rows owned by frequency group G of FS (bit i = row i).  Each
// group is closed under the (+p, -p) row pairs and covers whole float4s of
// frequencies: F(2) (T = 4, a row is one float4): rows {0, 3} (0 and infinity)
// and {1, 2} (+-1); F(5) (T = 7): rows {0..3} = frequencies 0..27 = float4s 0..6
// and rows {4,5,6} = float4s 7..12 (the last padded); F(6) (T = 8, a row is two
// float4s): rows {0,1,2,7} and {3,4,5,6}.
template <int M, int FS, int G>
constexpr unsigned group_rows() {
    static_assert(FS == 1 || (FS == 2 && M != 4), "frequency split built for F(2), F(5) and F(6)");
    if constexpr (FS == 1) return (1u << (M + 2)) - 1u;
    else if constexpr (M == 2) return G == 0 ? 0x9u : 0x6u;
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

// Waves synchronise through counters in LDS rather than workgroup barriers, so a
// consumer's epilogue never waits for the producers.  Every wait is bounded: it
// gives up after kSpinLimit polls (a broken handshake then ends the kernel with
// wrong output instead of hanging the GPU) and records that in the plan's status
// word, which wino_conv_status reports.
constexpr unsigned kSpinLimit = 1u << 22;
constexpr unsigned kErrSpinGaveUp = 1u;

// One lane sets the bit with an agent-scope atomic OR (a vector-memory atomic).
__device__ __forceinline__ void report_gave_up(unsigned *err) {
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_or(err, kErrSpinGaveUp, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Waits until counter c (in LDS, only growing) reaches target.
__device__ __forceinline__ void wait_at_least(const unsigned *c, unsigned target, unsigned *err) {
    for (unsigned n = 0; n < kSpinLimit; ++n) {
        if (__hip_atomic_load(c, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_WORKGROUP) >= target) return;
        __builtin_amdgcn_s_sleep(1);
    }
    report_gave_up(err);
}

// Stage ring: per LDS buffer (slot) a count of producer waves that have filled it
// and of consumer waves that have drained it, both only growing.  The g-th
// filling of a slot is complete when its fill count reaches 4(g+1); the slot may
// be filled again once its drain count reaches 4(g+1).
// Three slots where they fit (the producers may then run two stages ahead), two
// for F(5) and F(6).
template <int M>
constexpr int ws_slots() { return M <= 4 ? 3 : 2; }

// One wave's +1 on counter c, ordered after all of the wave's LDS accesses.
__device__ __forceinline__ void signal_wave(unsigned *c) {
    if ((threadIdx.x & 63) == 0) __hip_atomic_fetch_add(c, 1u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
}

// Items of a persistent workgroup: first + i * stride, i < count.  Each XCD takes
// one contiguous range of the items and its workgroups take items from it
// round-robin (workgroup b runs on XCD b % 8 as its (b / 8)-th workgroup), so the
// workgroups of an XCD work on neighbouring items at any time.
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

// Item numbering: with KM false the output-channel group varies fastest (items =
// tile groups x groups, the groups of one tile group adjacent: its input tiles
// are shared in L2); with KM true the tile group varies fastest (the tile groups
// of one output-channel group adjacent: its transformed kernels are shared in
// L2).  n_inner is the count of the fastest index.
template <bool KM>
__device__ __forceinline__ int item_tgroup(int it, int n_inner) { return KM ? it % n_inner : it / n_inner; }
template <bool KM>
__device__ __forceinline__ int item_kgroup(int it, int n_inner) { return KM ? it / n_inner : it % n_inner; }

// Work of one persistent workgroup, as one sequence of (item, channel stage)
// pairs shared by its producers and consumers: first its whole items (taken as by
// item_range from the first n_whole items), then its pieces of split items.  Each
// split item is cut into P pieces of L consecutive channel stages (the last one
// shorter when L does not divide the stages); the pieces ("split units", unit u is
// piece u % P of split item u / P) are distributed as by item_range.  Splitting
// only the items of a last, partly filled round spreads that round over compute
// units that would otherwise idle; splitting every item computes the layer as P
// convolutions over subsets of the input channels whose outputs are added (Sec.
// 7).  A piece yields a partial output, and the partial outputs of an item are
// added by whichever of its P contributors finishes last.
struct WsSplit {
    int n_whole;          // items distributed whole (item_range over the first n_whole)
    int tail_first;       // first split item
    int n_units;          // split items x P
    int P;                // pieces per split item (contributors)
    int piece;            // stages per piece (L)
    float *part;          // partial outputs, [split item][contributor][part_floats]
    unsigned *cnt;        // contributors arrived, per split item (zero between calls)
    int part_floats;      // floats of one partial output
    unsigned *err;        // plan's status word (bits set by waits that gave up)
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

// Blocking of one instantiation: R tiles and Kit output channels per item.
template <int M, int TB, int FS, int CSP>
struct WsShape {
    static constexpr int T = M + 2, T2 = T * T, F4 = freq_quads<M>();
    static constexpr int R = 16 * TB;          // tiles per item
    static constexpr int CC = 256 / R;         // input channels per stage
    static constexpr int SS = CC / 4;          // 4-channel matrix-core steps per stage
    static constexpr int SW = SS / CSP;        // steps of a stage one consumer multiplies
    static constexpr int P = FS * CSP;         // consumers per output block
    static constexpr int KBW = 4 / P;          // 16-channel output blocks per item
    static constexpr int KIT = 16 * KBW;       // output channels per item
    static constexpr int BUF = F4 * CC * R;    // float4s of one stage buffer
    static constexpr int NSLOT = ws_slots<M>();
    static constexpr int MM = M * M;
    static constexpr int MMP = (MM + 3) / 4 * 4;  // output tile padded to whole float4s
    // combine slots: P - 1 per output block, one output tile (MM floats) per lane
    static constexpr int NCOMB = (P - 1) * KBW * MM * 64;
    static_assert(4 % P == 0 && SS % CSP == 0 && SW % 2 == 0, "consumer split of a stage");
};

// Consumer wave of the persistent kernel: the workgroup's segments, as one
// continuous sequence of stages shared with the producers.  kbl: output block of
// the item; H: channel-step part; member index J = H * FS + G within the block
// (J = 0 adds the partial outputs and stores y).
template <int M, int TB, int FS, int G, int CSP, int H, bool SPLIT, bool KM>
__device__ __forceinline__ void ws_consume(const floatx4 *lds, float *comb, unsigned *combc, unsigned *ring,
                                           unsigned *skc,  // shared memory, written by other waves
                                           const floatx4 *__restrict__ wt, float *__restrict__ y,
                                           const Geometry &g, const WsSeq &sq, const WsSplit &sp,
                                           int n_inner, int kbl, int lane, int vec, bool ystream) {
    using S = WsShape<M, TB, FS, CSP>;
    constexpr int T = S::T, R = S::R, CC = S::CC, SS = S::SS, SW = S::SW, BUF = S::BUF;
    constexpr int NSLOT = S::NSLOT, P = S::P, KBW = S::KBW, MM = S::MM, MMP = S::MMP;
    constexpr GroupF4<M, FS, G> gm{};
    constexpr int NF4 = gm.N;  // float4s of frequencies this wave multiplies
    constexpr unsigned ROWS = group_rows<M, FS, G>();
    static_assert(gm.whole() && rows_pair_closed<M, ROWS>(), "groups split on float4 and pair bounds");
    const long long HW = (long long)g.H * g.W;
    const int32x4 yrs = make_rsrc(y, (unsigned)((long long)g.N * g.K * HW * 4));
    const unsigned hwb = (unsigned)(HW * 4), rowb = (unsigned)g.W * 4u;
    constexpr int J = H * FS + G;

    // Kernel operands alternate between two register sets over the wave's
    // channel steps (set a for even steps, b for odd ones): the loads of step u+1
    // are issued before the products of step u.  Every stage runs all its steps:
    // channels past C hold zero input tiles in LDS (and their operand indices are
    // clamped to the last step), so a segment's step sequence has an even length
    // and the loads past its end fetch the next segment's first steps, which
    // arrive during the epilogue.  The loads are unconditional, so that the wait
    // for an operand never has to include loads issued after it.
    // Operands are read with buffer loads: the lane's offset in a VGPR, the
    // (uniform) offset of a step of the wave's output block in an SGPR.
    kbl = __builtin_amdgcn_readfirstlane(kbl);
    constexpr unsigned SB = S::F4 * 1024u;  // bytes of one channel step of one output block
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
        const int c0 = sb * SS + H * SW;
        const unsigned cc0 = (unsigned)(c0 < last ? c0 : last);
#pragma unroll
        for (int lf = 0; lf < NF4; ++lf) wa[lf] = wload(wbase(item) + cc0 * SB, lf);
    }

    int q = 0;         // position in the stage sequence (selects the LDS buffer)
    unsigned seq = 0;  // partial tiles exchanged so far by this output block (P > 1)
    unsigned nsk = 0;  // partial-output epilogues so far
    int slot = 0;      // LDS buffer of stage q
    unsigned gen = 0;  // fillings of that buffer before stage q
    for (int k = 0; k < nseg; ++k) {
        if (k > 0) sq.segment(k, item, sb, se);
        int item2, sb2, se2;
        sq.segment(k + 1, item2, sb2, se2);
        const int nsteps = (se - sb) * SW;
        const unsigned bk = wbase(item), bn = wbase(item2);
        // operands of the wave's step u of this segment (u >= nsteps: the next segment's)
        auto wsrc = [&](int u) {
            const bool cur = u < nsteps;
            const int uu = cur ? u : u - nsteps;
            int c = ((cur ? sb : sb2) + uu / SW) * SS + H * SW + uu % SW;
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
        for (int jst = 0; jst < se - sb; ++jst, ++q) {
            wait_at_least(ring + slot, 4u * (gen + 1), sp.err);  // the producers have filled it
            const floatx4 *cur = lds + slot * BUF;
#pragma unroll
            for (int s = 0; s < SW; s += 2) {
                const int u = jst * SW + s;
                load_w(wb, wsrc(u + 1));
                __builtin_amdgcn_sched_barrier(0);
                step(wa, cur, H * SW + s);
                load_w(wa, wsrc(u + 2));
                __builtin_amdgcn_sched_barrier(0);
                step(wb, cur, H * SW + s + 1);
            }
            signal_wave(ring + NSLOT + slot);  // drained
            if (++slot == NSLOT) {
                slot = 0;
                ++gen;
            }
        }

        // Output transform Y = A^T Mm A per (output channel, tile) over this wave's
        // frequencies and channel steps; with P > 1 the block's partial tiles are
        // added; emit(t, v, k, ti, yy) consumes each finished output tile.
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
                    if constexpr (P > 1) {
                        // members j >= 1 write their partial into slot j - 1 of the
                        // block; member 0 adds them in member order (a fixed order,
                        // so results are reproducible) and stores
                        float *slots = comb + (long long)kbl * (P - 1) * MM * 64 + lane;
                        unsigned *written = combc + 2 * kbl, *readc = combc + 2 * kbl + 1;
                        if constexpr (J != 0) {
                            wait_at_least(readc, seq, sp.err);  // the slot's previous partial has been read
                            float *cs = slots + (J - 1) * MM * 64;
#pragma unroll
                            for (int e = 0; e < MM; ++e) cs[e * 64] = yy[e];
                            signal_wave(written);
                        } else {
                            wait_at_least(written, (unsigned)(P - 1) * (seq + 1), sp.err);
#pragma unroll
                            for (int jm = 0; jm < P - 1; ++jm)
#pragma unroll
                                for (int e = 0; e < MM; ++e) yy[e] += slots[jm * MM * 64 + e * 64];
                            __hip_atomic_store(readc, seq + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
                        }
                        ++seq;
                    }
                    if constexpr (J == 0) emit(t, v, kb * 16 + (lane >> 4) * 4 + v, ti, yy);
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
            if constexpr (J == 0) {
                // the KBW storing waves of the workgroup: written counts their
                // finished partials, wave kbl == 0 counts the workgroup's arrival
                unsigned *written = skc, *decided = skc + 1, *flag = skc + 2;
                asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // this wave's partial is stored
                signal_wave(written);
                if (kbl == 0) {
                    wait_at_least(written, (unsigned)KBW * (nsk + 1), sp.err);
                    if (lane == 0) {
                        const unsigned old = __hip_atomic_fetch_add(sp.cnt + t_split, 1u, __ATOMIC_RELAXED,
                                                                    __HIP_MEMORY_SCOPE_AGENT);
                        const unsigned is_last = (old + 1 == (unsigned)ncontrib) ? 1u : 0u;
                        if (is_last) __hip_atomic_store(sp.cnt + t_split, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        flag[nsk & 1u] = is_last;
                    }
                    signal_wave(decided);
                }
                wait_at_least(decided, nsk + 1, sp.err);
                if (__builtin_amdgcn_readfirstlane(flag[nsk & 1u]) != 0) sum_partials(pbase, ncontrib);
            }
            ++nsk;
        }

        // next segment's first operands are in wa (loaded as the wave's step nsteps)
    }
}

// Persistent warp-specialised fused kernel: one workgroup per compute unit
// (register and LDS use allow one).  The whole items of a workgroup come from
// one contiguous range per XCD, taken round-robin by its workgroups, so at any
// time the workgroups of an XCD work on neighbouring items: the groups that
// re-read one tile group's input, and the tile groups whose input tiles share
// halo rows and columns, find those in the XCD's L2.  The remaining items are
// split stage-wise across all workgroups (WsSeq).  Each workgroup runs its stages
// as one sequence, so the next item's first input tiles load and transform while
// the consumers finish the current item's output transform and stores.
template <int M, int TB, int FS, int CSP, bool VX, bool SPLIT, bool KM>
__global__ void __launch_bounds__(512) fused_ws_kernel(const float *__restrict__ x,
                                                       const floatx4 *__restrict__ wt,
                                                       float *__restrict__ y, Geometry g, int vec,
                                                       int n_inner, int n_items, WsSplit sp, int ystream) {
    using S = WsShape<M, TB, FS, CSP>;
    constexpr int T2 = S::T2, R = S::R, CC = S::CC, BUF = S::BUF, NSLOT = S::NSLOT, P = S::P;
    constexpr int COMB = (S::NCOMB + 3) / 4;     // float4s of the combine slots
    constexpr int NCNT = 2 * NSLOT + 4 + 2 * S::KBW;  // ring, split-output and combine counters
    constexpr int RING = (NCNT + 3) / 4;         // float4s of the counters
    __shared__ floatx4 lds[NSLOT * BUF + COMB + RING];
    float *comb = reinterpret_cast<float *>(lds + NSLOT * BUF);
    unsigned *ring = reinterpret_cast<unsigned *>(lds + NSLOT * BUF + COMB);  // fill counts, then drain counts
    unsigned *skc = ring + 2 * NSLOT;   // split outputs: written, decided, flag[2]
    unsigned *combc = skc + 4;          // per output block: partials written, rounds read

    const int tid = threadIdx.x;
    const int wave = tid >> 6;
    const int lane = tid & 63;
    if (tid < NCNT) ring[tid] = 0u;
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
        // flight where registers allow (m = 4), else PD = 1; F(2)'s 16-float tiles
        // allow PD = 4, so that the loads of a 64-channel item are all in flight
        // at once (measured on the 56x56 N=1 layer: 8.4 -> 7.9 us; larger F(2)
        // layers within 1 %).
        constexpr int PD = (M == 2) ? 4 : (M <= 4) ? 2 : 1;
        // The loads of round r + PD are issued unconditionally (past the last stage
        // they address tiles outside every image: no memory access), so that the
        // wait for a stage's data never has to cover loads issued after it.
        auto round = [&](int r, float *dcur, unsigned fcur, float *dnext, unsigned &fnext) {
            load_stage(dnext, fnext);
            if (r < nrounds) {
                const int slot = r % NSLOT;
                const unsigned gen = (unsigned)(r / NSLOT);
                if constexpr (VX) RowTile<M>::finish(dcur, fcur, maskcols);
                if (gen > 0) wait_at_least(ring + NSLOT + slot, 4u * gen, sp.err);
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
        } else if constexpr (PD == 2) {
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
        } else {
            // PD + 1 register sets rotating over the rounds (round r transforms set
            // r % (PD + 1) and loads into the set of round r + PD), the loop
            // unrolled by PD + 1 so that every set is named statically
            float d[PD + 1][T2];
            unsigned f[PD + 1] = {};
#pragma unroll
            for (int k = 0; k < PD; ++k) load_stage(d[k], f[k]);
            for (; r + PD < nrounds; r += PD + 1) {
#pragma unroll
                for (int k = 0; k <= PD; ++k) round(r + k, d[k], f[k], d[(k + PD) % (PD + 1)], f[(k + PD) % (PD + 1)]);
            }
#pragma unroll
            for (int k = 0; k < PD; ++k)
                if (r + k < nrounds) round(r + k, d[k], f[k], d[(k + PD) % (PD + 1)], f[(k + PD) % (PD + 1)]);
        }
        return;
    }

    // ---------------- consumers ----------------
    // wave w: output block w / P of the item, member j = w % P of the block, its
    // frequency group G = j % FS and channel-step part H = j / FS
    const int kbl = wave / P;
    const int jm = wave % P;
    const bool ys = ystream != 0;
#define WINO_WS_CONSUME(G_, H_)                                                                            \
    ws_consume<M, TB, FS, G_, CSP, H_, SPLIT, KM>(lds, comb, combc, ring, skc, wt, y, g, sq, sp, n_inner, kbl, \
                                                  lane, vec, ys)
    if constexpr (P == 1) {
        WINO_WS_CONSUME(0, 0);
    } else if constexpr (FS == 2 && CSP == 1) {
        if (jm == 0) WINO_WS_CONSUME(0, 0);
        else WINO_WS_CONSUME(1, 0);
    } else if constexpr (FS == 1 && CSP == 2) {
        if (jm == 0) WINO_WS_CONSUME(0, 0);
        else WINO_WS_CONSUME(0, 1);
    } else {
        static_assert(FS == 2 && CSP == 2, "consumer splits built: FS, CSP in {1, 2}");
        if (jm == 0) WINO_WS_CONSUME(0, 0);
        else if (jm == 1) WINO_WS_CONSUME(1, 0);
        else if (jm == 2) WINO_WS_CONSUME(0, 1);
        else WINO_WS_CONSUME(1, 1);
    }
#undef WINO_WS_CONSUME
}

// Split plan (see WsSeq): grid size, whole items per workgroup, the split items
// and the partial-output buffer they need.  csplit > 1 splits every item into
// that many channel pieces (at most one per stage); otherwise only a last, partly
// filled round may be split.
template <int M, int TB, int FS, int CSP>
SplitInfo ws_split_info(const Geometry &g, int num_cus, int csplit) {
    using S = WsShape<M, TB, FS, CSP>;
    constexpr int R = S::R, CC = S::CC, KBW = S::KBW;
    SplitInfo si{};
    const int n_tgroups = (g.ntiles + R - 1) / R;
    si.n_kgroups = (g.Kb + KBW - 1) / KBW;
    si.n_items = n_tgroups * si.n_kgroups;
    si.stages = (g.C + CC - 1) / CC;
    const int cus = num_cus < 1 ? 1 : num_cus;
    si.nfull = si.n_items / cus;
    si.grid = si.n_items < cus ? si.n_items : cus;
    si.part_floats = KBW * TB * 4 * S::MMP * 64;  // output tiles padded to float4s
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
    // dividing the stages, each piece at least 8 stages long) when at least half
    // of the compute units would idle in it otherwise.  A piece costs its
    // workgroup a partial-output epilogue (output transform, device-coherent
    // stores, arrival count) and the last contributor a sum of coherent reloads,
    // a fixed latency of several microseconds, so only long items gain
    // (measured: the 14x14 C=K=512 layer's 64-item last round of 32-stage items
    // split 4 ways, 344 -> 292 us at F(6); the 56x56 N=1 layer's 26 items of 4
    // stages split 4 ways, 14.5 -> 17.9 us; the 28x28 layer's 136-item last round
    // split 3 ways, 52.5 -> 79 us).  With four or more full rounds the imbalance
    // is small and items stay whole.
    constexpr int kMaxPieces = 4, kMaxSplitRounds = 4, kMinPieceStages = 8;
    const int tail = si.n_items - si.nfull * cus;
    if (si.nfull >= kMaxSplitRounds || tail == 0 || 2 * tail > cus) return si;
    int P = cus / tail < kMaxPieces ? cus / tail : kMaxPieces;
    while (P > 1 && (si.stages % P != 0 || si.stages / P < kMinPieceStages)) --P;
    if (P < 2) return si;
    si.tail_first = si.nfull * cus;
    si.n_tail = tail;
    si.piece = si.stages / P;
    si.n_units = tail * P;
    si.maxc = P;
    si.grid = si.nfull > 0 ? cus : tail * P;
    return si;
}

// Launch of one instantiation; returns the launch status.
template <int M, int TB, int FS, int CSP>
hipError_t launch_ws_t(const Geometry &g, const float *x, const float *wt, float *y, bool vec, int num_cus,
                       int csplit, const SplitBuffers &sb, hipStream_t s) {
    const SplitInfo si = ws_split_info<M, TB, FS, CSP>(g, num_cus, csplit);
    WsSplit sp;
    sp.n_whole = si.tail_first;
    sp.tail_first = si.tail_first;
    sp.n_units = si.n_units;
    sp.P = si.maxc;
    sp.piece = si.piece;
    sp.part = sb.part;
    sp.cnt = sb.cnt;
    sp.part_floats = si.part_floats;
    sp.err = sb.err;
    dim3 block(512), grid((unsigned)si.grid);
    // row-vector input loads need every row start aligned to the vector width
    // (m = 5: 4-byte aligned vector loads)
    const unsigned vw = (M == 4) ? 16u : (M == 5) ? 4u : 8u;
    const bool vx = (reinterpret_cast<uintptr_t>(x) % vw == 0) && ((unsigned)g.W * 4u) % vw == 0;
    // Item order: when the transformed kernels outweigh the input (deep layers),
    // the tile groups of one output-channel group are numbered adjacently, so the
    // workgroups of an XCD share that group's transformed kernels in L2.
    const bool km = si.n_kgroups > 1 && (double)g.T2 * g.C * g.K > (double)g.N * g.C * g.H * g.W;
    const int n_inner = km ? si.n_items / si.n_kgroups : si.n_kgroups;
    const int ystream = (long long)g.N * g.K * g.H * g.W * 4 >= kStreamOutputBytes ? 1 : 0;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, grid, block, 0, s, x, reinterpret_cast<const floatx4 *>(wt), y, g, vec ? 1 : 0,
                           n_inner, si.n_items, sp, ystream);
    };
    // layers whose items all stay whole run an instantiation without the split path
    const bool split = si.n_tail > 0;
#define WINO_WS_GO(VX_, SP_)                                                 \
    (km ? go(fused_ws_kernel<M, TB, FS, CSP, VX_, SP_, true>)                \
        : go(fused_ws_kernel<M, TB, FS, CSP, VX_, SP_, false>))
    if (vx) {
        if (split) WINO_WS_GO(true, true);
        else WINO_WS_GO(true, false);
    } else {
        if (split) WINO_WS_GO(false, true);
        else WINO_WS_GO(false, false);
    }
#undef WINO_WS_GO
    return hipGetLastError();
}

}  // namespace wino
