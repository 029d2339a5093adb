// Internal declarations shared by the host library (wino_api.cpp) and the
// kernels (wino_kernels.hip).  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <cstddef>
#include <cstdint>

namespace wino {

// Problem geometry and device buffers of one plan.
struct Geometry {
    int N, C, K, H, W, m;
    int T, T2;          // input tile edge m + 2 and frequencies T^2 (FFT: 16 and 16 * 9)
    int TH, TW;         // tiles per column / row: ceil(H/m), ceil(W/m)
    int ntiles;         // N * TH * TW
    int Cs;             // channel steps of 4 (matrix-core reduction depth): ceil(C/4)
    int Kb;             // output-channel blocks of 16: ceil(K/16)
    int Kb_alloc;       // Kb rounded up to a multiple of 4 (padding blocks are zero)
    int tiles_p;        // ntiles rounded up to a multiple of 64 (three-stage buffers)
};

// Blocking of the fused kernel (the paper's task, Sec. 4.1): R tiles and kit
// output channels per work item; the input channels of a stage are 256 / R (one
// (tile, channel) pair per producer lane).
struct FusedCfg {
    int R;         // tiles per item: 16 or 32
    int kit;       // output channels per item: 16, 32 or 64
    int num_cus;   // compute units of the device (persistent grid size)
    int csplit;    // channel pieces per work item (0 or 1: whole items)
};

// The (m, R, kit) blockings the fused kernel is built for, with the kernel
// template of each: X(m, R, kit, TB, FS, CSP), R = 16 TB tiles, FS * CSP consumer
// waves per 16-channel output block (wino_ws.h).  The build compiles
// wino_fused_inst.hip once per entry.
#define WINO_FUSED_BLOCKINGS(X)                                                                \
    X(2, 32, 64, 2, 1, 1) X(2, 16, 64, 1, 1, 1) X(2, 32, 32, 2, 2, 1) X(2, 16, 32, 1, 1, 2)     \
    X(2, 16, 16, 1, 2, 2) X(4, 16, 64, 1, 1, 1) X(4, 16, 32, 1, 1, 2) X(5, 16, 32, 1, 2, 1)     \
    X(5, 16, 16, 1, 2, 2) X(6, 16, 32, 1, 2, 1) X(6, 16, 16, 1, 2, 2)

struct FusedBlocking {
    int m, R, kit;
    int tb, fs, csp;
};
#define WINO_FB_ENTRY(m, R, kit, tb, fs, csp) {m, R, kit, tb, fs, csp},
constexpr FusedBlocking kFusedBlockings[] = {WINO_FUSED_BLOCKINGS(WINO_FB_ENTRY)};
#undef WINO_FB_ENTRY
bool fused_blocking_built(int m, int R, int kit);

// Split plan of the warp-specialised fused kernel: the last round of items (or,
// with channel splitting, every item) is divided stage-wise among workgroups;
// each split item's partial outputs go to a plan-owned buffer and are added by
// the contributor that finishes last.
struct SplitInfo {
    int grid;              // workgroups launched
    int n_items, n_kgroups, stages;
    int nfull;             // full rounds of whole items (n_items / grid)
    int tail_first, n_tail;  // items [0, tail_first) are whole, the n_tail after are split
    int n_units;           // n_tail * maxc pieces
    int piece;             // stages per piece of a split item (the last piece may be shorter)
    int maxc;              // contributors (pieces) per split item
    int part_floats;       // floats of one contributor's partial output
};
struct SplitBuffers {
    float *part;           // n_tail * maxc * part_floats floats
    unsigned *cnt;         // n_tail arrival counters, zero between calls
    unsigned *err;         // status word: bits set by kernel waits that gave up
};
SplitInfo fused_split_info(const Geometry &g, const FusedCfg &cfg);

// One line naming the fused kernel a call launches and its blocking.
void describe_fused(const Geometry &g, const FusedCfg &cfg, char *buf, size_t len);

// Kernel transform: w (K x C x 3 x 3) -> wt in matrix-core operand order.  The
// first workgroup also sets the nzero words at zero to 0 (counters a following
// fused kernel needs cleared, without a memset).
hipError_t launch_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s,
                                   unsigned *zero = nullptr, int nzero = 0);

// Fused: x -> y with the transformed kernels wt.
hipError_t launch_fused(const Geometry &g, const FusedCfg &cfg, const float *x, const float *wt,
                        float *y, const SplitBuffers &sb, hipStream_t s);

// Three-stage: x -> U -> M -> y.
hipError_t launch_input_transform(const Geometry &g, const float *x, float *U, hipStream_t s);
hipError_t launch_frequency_gemm(const Geometry &g, const float *U, const float *wt, float *M,
                                 hipStream_t s);
hipError_t launch_output_transform(const Geometry &g, const float *M, float *y, hipStream_t s);

// FFT-tile algorithm (16 x 16 tiles, m = 14): kernel spectra, then the fused kernel.
hipError_t launch_fft_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s);
hipError_t launch_fft_fused(const Geometry &g, const float *x, const float *wt, float *y, hipStream_t s);

// Sets the message wino_last_error() returns on the calling thread (printf format).
void set_error(const char *fmt, ...);

// Host-side checks shared by the entry points (wino_api.cpp): geometry of a
// problem with overflow checks (WINO_OK or a WINO_E* status, message set); p
// (bytes long) a device allocation on `device` that holds it; a stream of
// `device` (NULL: the null stream); byte ranges overlapping.
int make_geometry(int N, int C, int K, int H, int W, int m, int algo, Geometry *g);
int check_device_ptr(const void *p, size_t bytes, int device, const char *name);
int check_stream_device(hipStream_t s, int device);
bool overlap(const void *a, size_t na, const void *b, size_t nb);

// Default blocking of a layer among the built ones (restricted to tiles per item
// want_R and output channels per item want_kit where those are nonzero).
FusedCfg fused_cfg_default(const Geometry &g, int num_cus, int want_R = 0, int want_kit = 0);

// One line naming the three-stage kernels.
void describe_three_stage(const Geometry &g, char *buf, size_t len);

}  // namespace wino
