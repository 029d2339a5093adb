/*
 * wino_conv.h -- C ABI of a fused Winograd 3x3 convolution for AMD MI355X (gfx950).
 *
 * The operation (Sec. 2.1, Eq. 1, with the pad of 1 used in Sec. 6): for every
 * image n, output channel k and pixel (h, v),
 *
 *     y[n,k,h,v] = sum_{c<C} sum_{r<3} sum_{s<3} x[n,c,h+r-1,v+s-1] * w[k,c,r,s]
 *
 * with x read as zero outside the image (implicit padding), stride 1.  It is
 * computed as the Winograd F(m x m, 3 x 3) transformed convolution of Eq. 3,
 * y = A^T [ sum_c (G w G^T) (.) (B^T d B) ] A over overlap-add tiles of edge
 * T = m + 2 (Sec. 2.1), for m in {2, 4, 5, 6} (m = 5, T = 7, is the tile of the
 * paper's experiments, Sec. 6) and, with the three-stage algorithm only, m = 7
 * (T = 9: two tiles cover a 14-pixel image side exactly), or as the FFT-tile
 * convolution of the same sections with T = 16 (m = 14; Sec. 4 gives T >= 16 for
 * FFT).
 *
 * Layouts: x is N x C x H x W, w is K x C x 3 x 3, y is N x K x H x W, all dense
 * row-major fp32.  x, w and y are device pointers on the plan's device.
 *
 * Two algorithms compute the same result:
 *   WINO_ALGO_FUSED       one kernel per call does, for a block of tiles, the
 *                         input transform, the per-frequency products over C on
 *                         the matrix cores and the output transform, keeping the
 *                         transformed tiles on chip (Sec. 4, the "L3 fused" task
 *                         of R tiles).
 *   WINO_ALGO_THREE_STAGE the standard pipeline of Sec. 3: all input transforms
 *                         to device memory, T^2 products over C, then all output
 *                         transforms.
 *   WINO_ALGO_FFT         fused like WINO_ALGO_FUSED, with the 16 x 16 discrete
 *                         Fourier transform in place of the Winograd transforms
 *                         (m must be 14): per tile the 16 x 9 frequencies of the
 *                         half spectrum (the rest are complex conjugates,
 *                         Sec. 2.1), complex products over C against the
 *                         conjugated spectra of the zero-padded kernels (the
 *                         convolution theorem for the correlation above).
 * All first transform the kernels (Sec. 3, step 2: kernel matrices obtained by
 * transforming the kernels), unless the weights were set ahead of time with
 * wino_conv_set_weights.
 *
 * Errors: functions return WINO_OK (0) or a negative status; plan constructors
 * return NULL.  In every failure case wino_last_error() describes it.  Arguments
 * are checked before any GPU work is queued; the library never aborts, exits or
 * prints (unless the environment variable WINO_LOG=1, which logs plan choices to
 * stderr).  Not thread-safe per plan: one plan serves one stream at a time.
 */
#ifndef WINO_CONV_H
#define WINO_CONV_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct wino_plan wino_plan; /* opaque */

enum {
    WINO_OK = 0,
    WINO_EINVAL = -1,       /* bad argument */
    WINO_EUNSUPPORTED = -2, /* valid request this library does not handle */
    WINO_ENOMEM = -3,       /* device allocation failed */
    WINO_EHIP = -4,         /* a HIP call or kernel launch failed */
    WINO_EKERNEL = -5       /* a kernel reported a failure through the plan's status word */
};

enum {
    WINO_ALGO_FUSED = 0,
    WINO_ALGO_THREE_STAGE = 1,
    WINO_ALGO_FFT = 2
};

/* Intermediate buffers a plan owns (for wino_conv_copy_intermediate). */
enum {
    WINO_BUF_WEIGHTS = 0,   /* transformed kernels, see wino_conv_intermediate_dims */
    WINO_BUF_INPUT = 1,     /* three-stage only: transformed input tiles  */
    WINO_BUF_PRODUCT = 2    /* three-stage only: per-frequency products    */
};

/* Optional blocking of the fused algorithm (the task of Sec. 4.1: a workgroup
 * transforms R input tiles, multiplies them by the transformed kernels of a
 * group of output channels over all input channels, and inverse-transforms the
 * results, all on chip).  A field of 0 keeps the automatic choice.
 *   tiles_per_wg:   R, tiles per task: 16, or 32 for m = 2.
 *   k_per_wg:       output channels per task: 64, 32 or 16.  Built (m, R, k):
 *                   m = 2: (32, 64), (16, 64), (32, 32), (16, 32), (16, 16);
 *                   m = 4: (16, 64), (16, 32);  m = 5, 6: (16, 32), (16, 16).
 *                   The task's result matrices (R x k x T^2 floats) live in
 *                   registers, which bounds R * k (Sec. 4.1's private capacity).
 *   c_chunk:        input channels per pipeline stage; it is 256 / R (each of the
 *                   256 producer lanes transforms one (tile, channel) pair per
 *                   stage), so only 0 or that value is accepted.
 *   channel_splits: compute the layer as P convolutions over disjoint,
 *                   consecutive subsets of the input channels and add their
 *                   outputs (Sec. 7 on splitting channels; the output transform
 *                   is linear, so each subset's products are inverse-transformed
 *                   on their own).  Every work item is cut into pieces of
 *                   L = ceil(S / channel_splits) channel stages, S = ceil(C /
 *                   c_chunk), so P = ceil(S / L) pieces, at most S.  The pieces'
 *                   outputs go to a plan-owned buffer of P partial tiles per item
 *                   and are added in channel order by the piece that finishes last
 *                   (results do not depend on the order pieces run in, but differ
 *                   from the unsplit sum by rounding).  0 or 1: no split; at most
 *                   WINO_MAX_CHANNEL_SPLITS.
 * Automatic choice (wino_conv_plan): the largest task that fits (k at its
 * maximum, R = 32 for m = 2 with C <= 64, else 16: most reuse of each
 * transformed input tile and transformed-kernel operand) as long as the layer has
 * at least one task per compute unit; otherwise the blocking with the most
 * tasks.  wino_conv_plan_tuned measures every blocking instead. */
#define WINO_MAX_CHANNEL_SPLITS 64
typedef struct {
    int tiles_per_wg;
    int k_per_wg;
    int c_chunk;
    int channel_splits;
} wino_tuning;

/* Create a plan for an F(m x m, 3 x 3) convolution of an N x C x H x W input
 * with K output channels, on the current HIP device, with the fused algorithm
 * and automatic blocking.  Allocates the plan's device workspace: the
 * transformed kernels (T^2 * C * K floats rounded up to the blocking) and, when
 * the last round of work items is split across compute units, their partial
 * outputs and arrival counters (zeroed here; every call leaves them zero).
 * Returns NULL (see wino_last_error) if a size is < 1, m is not 2, 4, 5 or 6 (also 7
 * for WINO_ALGO_THREE_STAGE; 14 for WINO_ALGO_FFT, which takes no other m), a
 * size overflows the 32-bit offsets the kernels use (each of x and y must be
 * below 2^31 bytes), or the allocation fails. */
wino_plan *wino_conv_plan(int N, int C, int K, int H, int W, int m);

/* As wino_conv_plan, choosing the algorithm (WINO_ALGO_*) and optional blocking
 * overrides (t may be NULL; they apply to WINO_ALGO_FUSED and are ignored by the
 * others, except that channel_splits > 1 is refused for them).  The
 * three-stage plan also allocates its intermediate buffers (T^2 * tiles * (C + K)
 * floats, rounded up to the blocking); the FFT plan's transformed kernels take
 * 144 * 16 bytes per (input, output) channel pair, padded to multiples of 4 and
 * 16. */
wino_plan *wino_conv_plan_ex(int N, int C, int K, int H, int W, int m, int algo,
                             const wino_tuning *t);

/* Queue y = conv(x, w) on stream (a hipStream_t; NULL is the null stream).
 * Asynchronous: returns once the work is queued; synchronise the stream before
 * reading y.  y is fully overwritten.  x, w and y must be device allocations on
 * the plan's device large enough for their tensors, 4-byte aligned, and y must
 * not overlap x or w.  Returns WINO_EINVAL for a NULL plan or pointer, a bad
 * pointer, overlap, or a stream of another device; WINO_EHIP if a launch fails. */
int wino_conv_run(const wino_plan *p, const float *x, const float *w, float *y, void *stream);

/* Steady-state inference (Sec. 3 footnote: kernels transformed ahead of time):
 * transform w (K x C x 3 x 3, device) into the plan's workspace on stream. */
int wino_conv_set_weights(wino_plan *p, const float *w, void *stream);

/* Queue y = conv(x, w) with the kernels most recently transformed into the plan
 * (by wino_conv_set_weights or wino_conv_run), skipping the kernel transform.
 * Returns WINO_EINVAL if the plan holds no kernels yet, otherwise as wino_conv_run. */
int wino_conv_run_pretransformed(const wino_plan *p, const float *x, float *y, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): y = conv(x, w) as
 * wino_conv_run does it with a fused plan of automatic blocking (kernel transform,
 * then the fused kernel; the same kernels, so the same bits), without a plan and
 * without allocating.  The scratch the fused path needs -- the transformed
 * kernels (T^2 * C * K floats rounded up to the blocking), the split items'
 * partial outputs and arrival counters -- lives in a file-scope device array of
 * WINO_NOALLOC_SCRATCH_BYTES, one per GPU, held until the process ends; the
 * counters are cleared by the kernel transform at every call (no memset).
 * Every call on a GPU shares that GPU's array and leaves its own contents in it:
 * calls that overlap on one GPU (different streams or threads) race and give
 * wrong results; order them on one stream.  Layers whose scratch exceeds the
 * array (for example C = K = 512 at F(6x6,3x3): 67 MB of transformed kernels)
 * return WINO_EUNSUPPORTED before any HIP call when the transformed kernels alone
 * do not fit, otherwise before any launch; use a plan for them.
 * x, w, y as for wino_conv_run (device pointers on the current device).  status:
 * NULL, or a device word into which the fused kernel ORs the bits of a bounded
 * wait that gave up (as wino_conv_status reports them for plans; never cleared
 * here, so a caller can check it after many calls).  Asynchronous on stream.
 * Returns WINO_OK, WINO_EINVAL (bad sizes, m, pointer or stream),
 * WINO_EUNSUPPORTED (too large), WINO_EHIP (a HIP call or launch failed). */
#define WINO_NOALLOC_SCRATCH_BYTES (16u << 20)
int wino_conv_run_noalloc(int N, int C, int K, int H, int W, int m, const float *x, const float *w,
                          float *y, unsigned *status, void *stream);

/* Free the plan and its device memory.  NULL is ignored.  The caller must make
 * sure no queued work still uses the plan. */
void wino_conv_destroy(wino_plan *p);

/* Bytes of device workspace the plan holds (0 for NULL). */
size_t wino_conv_workspace_bytes(const wino_plan *p);

/* Sizes of the problem: number of tiles N*ceil(H/m)*ceil(W/m), direct-convolution
 * flops 2*N*C*K*H*W*9 and transform-domain flops 2*T^2*tiles*C*K (FFT:
 * 8*144*tiles*C*K, four real multiply-adds per complex one at each of the 144
 * kept frequencies).  Any output pointer may be NULL.  Returns WINO_EINVAL for
 * a NULL plan. */
int wino_conv_info(const wino_plan *p, long long *n_tiles, double *direct_flops,
                   double *tdomain_flops);

/* Logical layout of an intermediate buffer as up to 4 dims (outermost first,
 * unused trailing dims are 1), for tests that read it back:
 *   WINO_BUF_WEIGHTS: [Kb][Cs][Q][64][4], Q = ceil(T^2/4): element (f, c, k) of
 *                     G w[k,c] G^T sits at kb = k/16, cs = c/4, block f/4, lane
 *                     (c%4)*16 + k%16, slot f%4 (the matrix-core operand order);
 *                     slots past f = T^2 - 1 (F(5)) hold zeros.  Dims returned:
 *                     {Kb, Cs, 4*Q, 64} with f in the third dim as described.
 *                     FFT plans: [Cs][Kb][144][64][4], element (f, c, k) at cs =
 *                     c/4, kb = k/16, frequency f = p*9 + q (spectrum row p,
 *                     column q <= 8), lane (c%4)*16 + k%16, holding {Re, Im,
 *                     -Im, 0} of the spectrum of w[k,c] zero-padded to 16 x 16;
 *                     dims returned {Cs, Kb, 144, 256}.
 *   WINO_BUF_INPUT:   three-stage plans only: [F4][TB][Cs][64][4], F4 =
 *                     ceil(T^2/4), TB = tiles rounded up to 64, / 16: element
 *                     (f, c, t) of U = B^T d B at f4 = f/4, tb = t/16, cs = c/4,
 *                     lane (c%4)*16 + t%16, slot f%4.  Dims {F4, TB, Cs, 256}.
 *   WINO_BUF_PRODUCT: three-stage plans only: [F4][TB][Kb][4][64][4], Kb =
 *                     ceil(K/16) rounded up to 4: element (f, k, t) of
 *                     M = sum_c W' U at f4 = f/4, tb = t/16, kb = k/16, v = k%4,
 *                     lane ((k%16)/4)*16 + t%16, slot f%4.  Dims {F4, TB, Kb, 1024}.
 *                     Channels, output channels, tiles and frequencies past the
 *                     problem hold zeros.
 * Frequency f = i*T + j for transform row i, column j; tile t = (n*TH + ty)*TW + tx. */
int wino_conv_intermediate_dims(const wino_plan *p, int which, long long dims[4]);

/* Copy an intermediate buffer to host memory (count floats, synchronous on the
 * null stream after a device synchronisation).  Returns WINO_EINVAL if the plan
 * has no such buffer or count is larger than it. */
int wino_conv_copy_intermediate(const wino_plan *p, int which, float *host_dst, size_t count);

/* Synchronous check of the plan's status word.  The persistent fused kernel's
 * producer and consumer waves hand stages to each other through counters in
 * shared memory; every wait is bounded (it gives up after about 4 million polls
 * rather than hang the GPU), and a wait that gives up sets a bit in a device word
 * the plan owns.  A call whose wait gave up has queued without error but its y is
 * not valid.  This function waits for all work on the device
 * (hipDeviceSynchronize), reads the word, and if it is nonzero clears it and the
 * plan's split arrival counters and returns WINO_EKERNEL (wino_last_error names
 * the bits); otherwise WINO_OK.  WINO_EINVAL for a NULL plan, WINO_EHIP if a HIP
 * call fails. */
int wino_conv_status(const wino_plan *p);

/* Test hook for the status plumbing: writes `word` into the plan's status word
 * (synchronous copy), as a kernel whose wait gave up would.  Returns WINO_OK,
 * WINO_EINVAL for a NULL plan, WINO_EHIP if the copy fails. */
int wino_conv_debug_set_status(const wino_plan *p, unsigned word);

/* One line of text naming the kernel(s) a call of the plan launches and their
 * blocking: for the fused algorithm the kernel and its template parameters, the
 * tiles per task R and output channels per task, channels per stage, work items,
 * grid and split pieces; for the three-stage algorithm its three kernels.  The
 * text (NUL-terminated, truncated to len - 1 characters) goes to buf.  Returns
 * WINO_EINVAL for a NULL plan or buffer or len == 0. */
int wino_conv_describe(const wino_plan *p, char *buf, size_t len);

/* Message describing the last failure on the calling thread ("" if none). */
const char *wino_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* WINO_CONV_H */
