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

// Fused-kernel schedule and blocking.
enum { kSchedShared = 1, kSchedPerWave = 2, kSchedSpecialised = 3, kSchedPersistent = 4 };
struct FusedCfg {
    int schedule;  // kSchedShared, kSchedPerWave, kSchedSpecialised or kSchedPersistent
    int tb;        // shared: tile blocks of 16 per workgroup
    int nkb;       // per-wave: 16-channel output blocks per wave
    int waves;     // per-wave: waves per workgroup (each owns 16 tiles)
    int num_cus;   // compute units of the device (persistent grid size)
    int csplit;    // specialised: channel pieces per work item (0 or 1: whole items)
};

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
};
SplitInfo fused_split_info(const Geometry &g, const FusedCfg &cfg);

// Kernel transform: w (K x C x 3 x 3) -> wt in matrix-core operand order.
hipError_t launch_weight_transform(const Geometry &g, const float *w, float *wt, hipStream_t s);

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

// Fused blocking the kernels are instantiated for, per m.
bool fused_cfg_supported(int m, const FusedCfg &cfg);
FusedCfg fused_cfg_default(const Geometry &g);

}  // namespace wino
