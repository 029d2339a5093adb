/*
 * wino_tune.h -- per-layer tuning of the Winograd convolution and its wisdom table.
 *
 * Sec. 6 runs one fixed configuration on every layer and notes that tuning the
 * parameters for each particular layer can only improve the results; Sec. 7
 * says that the parameters (R, the tiles per task, among them) can be tuned once
 * and stored in a wisdom file.  Here the tuned parameters are the tile size m of
 * F(m x m, 3 x 3), m in {2, 4, 5, 6} (the paper's T = m + 2), the fused kernel's
 * blocking at each m -- tiles per task R and output channels per task, every
 * blocking the kernel is built for (wino_fused_blockings) -- and, optionally,
 * the algorithm (three-stage at each m and at m = 7, or the FFT-tile algorithm
 * with m = 14).
 * A tuning result is remembered per (GPU architecture, compute units, N, C, K,
 * H, W, candidate set) in a process-wide wisdom table that can be written to and
 * read from a text file.
 *
 * Wisdom file: text, one entry per line, '#' starts a comment line:
 *     <arch> <cus> <N> <C> <K> <H> <W> <candidates> <m> <algo> <R> <k> <microseconds>
 * arch is the device's architecture name (e.g. gfx950), candidates is the
 * candidate mask in hexadecimal (0x...), algo is 0 (fused), 1 (three-stage) or
 * 2 (FFT, with m = 14), R and k the fused blocking (tiles and output channels per
 * task; 0 0 for the other algorithms) and microseconds the measured time per
 * call of back-to-back calls.
 *
 * Thread safety: the wisdom table is guarded by a lock; plans are as in
 * wino_conv.h (one stream at a time).
 */
#ifndef WINO_TUNE_H
#define WINO_TUNE_H

#include "wino_conv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Candidate mask bits: tile sizes, whether the three-stage algorithm is also
 * tried at each of them, and whether the FFT-tile algorithm is tried. */
enum {
    WINO_TUNE_M2 = 1 << 2,
    WINO_TUNE_M4 = 1 << 4,
    WINO_TUNE_M5 = 1 << 5,
    WINO_TUNE_M6 = 1 << 6,
    WINO_TUNE_M7 = 1 << 7,  /* three-stage only: needs WINO_TUNE_THREE_STAGE */
    WINO_TUNE_THREE_STAGE = 1 << 8,
    WINO_TUNE_FFT = 1 << 9  /* the FFT-tile algorithm (m = 14) */
};

/* A plan for the convolution of wino_conv_plan (N x C x H x W input, K output
 * channels) with the m, fused blocking and algorithm that run fastest on the
 * current device among the candidates (a nonzero mask of WINO_TUNE_* bits with at least one
 * WINO_TUNE_M* or the WINO_TUNE_FFT bit).  If the wisdom table holds the answer it is used directly;
 * otherwise every candidate is planned and timed here: its kernels transformed
 * once, at least 20 ms of back-to-back warm-up calls of
 * wino_conv_run_pretransformed (so that every candidate is timed at the shader
 * clock's working frequency), then the median time per call of 5 batches of at
 * least 1 ms of back-to-back calls, on device buffers of the layer's size that this function
 * allocates, fills with a constant and frees before returning (synchronous;
 * needs room for x, y and w beside the largest candidate's workspace).  The
 * result enters the wisdom table.  chosen_m, chosen_algo and call_us (each may
 * be NULL) receive the choice and its measured time (0 if it came from the
 * table without a time).  Returns NULL (see wino_last_error) for bad sizes, a
 * bad mask, or a failed allocation or launch. */
wino_plan *wino_conv_plan_tuned(int N, int C, int K, int H, int W, unsigned candidates,
                                int *chosen_m, int *chosen_algo, double *call_us);

/* The tile size m, algorithm and fused blocking (tiles and output channels per
 * task; 0 for the other algorithms) of a plan.  Any output pointer may be NULL.
 * Returns WINO_EINVAL for a NULL plan. */
int wino_conv_plan_params(const wino_plan *p, int *m, int *algo, int *tiles_per_wg, int *k_per_wg);

/* The fused blockings the library is built for: up to max (m, tiles_per_wg,
 * k_per_wg) triples are written to the arrays (each may be NULL); returns the
 * total number. */
int wino_fused_blockings(int *m, int *tiles_per_wg, int *k_per_wg, int max);

/* Look up an entry: on WINO_OK, *found is 1 and *m, *algo, *tiles_per_wg,
 * *k_per_wg hold the entry, or *found is 0.  arch is an architecture name as in
 * the file.  Returns WINO_EINVAL for NULL pointers. */
int wino_wisdom_lookup(const char *arch, int cus, int N, int C, int K, int H, int W,
                       unsigned candidates, int *found, int *m, int *algo, int *tiles_per_wg,
                       int *k_per_wg);

/* Write the table to path (replacing the file).  Returns WINO_EINVAL if the
 * file cannot be written. */
int wino_wisdom_save(const char *path);

/* Merge the entries of a wisdom file into the table (an entry replaces one
 * with the same key).  The file is checked completely first: a malformed line
 * (wrong field count or an m, algo or size out of range) leaves the table
 * unchanged and returns WINO_EINVAL naming the line; so does an unreadable
 * file. */
int wino_wisdom_load(const char *path);

/* Remove every entry.  Number of entries in the table. */
void wino_wisdom_clear(void);
int wino_wisdom_size(void);

#ifdef __cplusplus
}
#endif

#endif /* WINO_TUNE_H */
