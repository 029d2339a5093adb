/*
 * Direct 3x3 convolution, stride 1, zero padding 1, fp64 accumulation.
 * Oracle code: test infrastructure only, never part of the GPU library.
 *
 * It is Eq. 1 of the paper (Sec. 2.1), I'_{b,c'} = sum_c I_{b,c} * W_{c'c},
 * read as the cross-correlation that CNN layers compute (no kernel flip), with
 * the pad of 1 used in the paper's experiments (Sec. 6) and implicit zero
 * padding (Sec. 2.1: padding is not materialised):
 *
 *   y[n,k,h,v] = sum_{c<C} sum_{r<3} sum_{s<3} x[n,c,h+r-1,v+s-1] * w[k,c,r,s]
 *
 * where x is zero outside [0,H) x [0,W).  Layouts: x NCHW fp32, w KCRS fp32
 * (the paper's C' x C x K x K kernel tensor), y NKHW fp64.  The fp32 inputs are
 * promoted to fp64 and every sum is carried in fp64.
 *
 * Restricting h and v to the ranges where the input index is inside the image
 * is the same as multiplying by the zero padding; nothing else is reordered
 * beyond the choice of loop order.  OpenMP runs independent (n, k) planes in
 * parallel.
 */
#include <stdint.h>
#include <stddef.h>
#include <omp.h>

static void conv_plane(const float *x, const float *w, double *yp,
                       int64_t n, int64_t k, int64_t C, int64_t H, int64_t W)
{
    for (int64_t i = 0; i < H * W; ++i) yp[i] = 0.0;
    for (int64_t c = 0; c < C; ++c) {
        const float *xp = x + (n * C + c) * H * W;
        for (int r = 0; r < 3; ++r) {
            for (int s = 0; s < 3; ++s) {
                const double wv = (double)w[((k * C + c) * 3 + r) * 3 + s];
                /* output rows h with 0 <= h + r - 1 < H */
                const int64_t h0 = (r == 0) ? 1 : 0;
                const int64_t h1 = (r == 2) ? H - 1 : H;
                const int64_t v0 = (s == 0) ? 1 : 0;
                const int64_t v1 = (s == 2) ? W - 1 : W;
                for (int64_t h = h0; h < h1; ++h) {
                    const float *xrow = xp + (h + r - 1) * W + (s - 1);
                    double *yrow = yp + h * W;
                    for (int64_t v = v0; v < v1; ++v)
                        yrow[v] += (double)xrow[v] * wv;
                }
            }
        }
    }
}

/* Full output: y must hold N*K*H*W doubles.  Returns 0, or -1 on bad sizes. */
int oracle_direct_conv_f64(const float *x, const float *w, double *y,
                           int64_t N, int64_t C, int64_t K, int64_t H, int64_t W)
{
    if (N < 0 || C < 0 || K < 0 || H < 0 || W < 0) return -1;
    int64_t planes = N * K;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t p = 0; p < planes; ++p)
        conv_plane(x, w, y + p * H * W, p / K, p % K, C, H, W);
    return 0;
}

/* Selected output planes: plane i is (n_idx[i], k_idx[i]) and goes to
 * y + i*H*W.  Used to check full-size layers on a sample of their outputs.
 * Returns 0, or -1 on a bad size or an index out of range. */
int oracle_direct_conv_planes_f64(const float *x, const float *w, double *y,
                                  int64_t N, int64_t C, int64_t K, int64_t H, int64_t W,
                                  const int64_t *n_idx, const int64_t *k_idx, int64_t count)
{
    if (N < 0 || C < 0 || K < 0 || H < 0 || W < 0 || count < 0) return -1;
    for (int64_t i = 0; i < count; ++i)
        if (n_idx[i] < 0 || n_idx[i] >= N || k_idx[i] < 0 || k_idx[i] >= K) return -1;
    #pragma omp parallel for schedule(dynamic, 1)
    for (int64_t i = 0; i < count; ++i)
        conv_plane(x, w, y + i * H * W, n_idx[i], k_idx[i], C, H, W);
    return 0;
}

/* Number of OpenMP threads the entry points above use. */
int oracle_num_threads(void)
{
    return omp_get_max_threads();
}
