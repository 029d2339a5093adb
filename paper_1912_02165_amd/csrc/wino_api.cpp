// C ABI of the Winograd 3x3 convolution library (declared in include/wino_conv.h):
// plan construction, argument checks, workspace ownership and launch order.
#include "wino_conv.h"
#include "wino_internal.h"
#include "wino_tune.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>

using wino::FusedCfg;
using wino::Geometry;

struct wino_plan {
    Geometry g;
    int algo;
    FusedCfg fcfg;
    int device;
    float *wt;        // transformed kernels, matrix-core operand order
    size_t wt_bytes;
    float *U;         // three-stage: transformed input tiles  [F4][TB][Cs][64][4]
    float *Mf;        // three-stage: per-frequency sums       [F4][TB][Kb_alloc][4][64][4]
    size_t U_bytes, M_bytes;
    wino::SplitBuffers split;  // fused: partial outputs of split items and their counters
    size_t part_bytes, cnt_bytes;
    mutable bool weights_set; // wt holds transformed kernels (set_weights or the last run)
};

namespace {

thread_local std::string g_err;

void set_err(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
}

bool log_enabled() {
    const char *e = getenv("WINO_LOG");
    return e && e[0] == '1';
}

int hip_fail(const char *what, hipError_t e) {
    set_err("%s: %s", what, hipGetErrorString(e));
    return WINO_EHIP;
}

}  // namespace

// 64-bit geometry with overflow checks; fills g on success.
// Tiles of edge T = m + 2 (Winograd) or T = 16, m = 14 (FFT, whose T2 counts
// the 16 x 9 kept frequencies of a tile's half spectrum).
int wino::make_geometry(int N, int C, int K, int H, int W, int m, int algo, Geometry *g) {
    if (N < 1 || C < 1 || K < 1 || H < 1 || W < 1) {
        set_err("sizes must be >= 1 (N=%d C=%d K=%d H=%d W=%d)", N, C, K, H, W);
        return WINO_EINVAL;
    }
    if (algo == WINO_ALGO_FFT) {
        if (m != 14) {
            set_err("m=%d: the FFT algorithm uses 16 x 16 tiles, m = 14", m);
            return WINO_EINVAL;
        }
    } else if (m == 7) {
        if (algo != WINO_ALGO_THREE_STAGE) {
            set_err("m=7: F(7x7,3x3) runs on the three-stage algorithm only (its 81 frequencies per tile "
                    "and channel do not fit the fused kernel's LDS stage ring)");
            return WINO_EUNSUPPORTED;
        }
    } else if (m != 2 && m != 4 && m != 5 && m != 6) {
        set_err("m=%d: only F(2x2,3x3), F(4x4,3x3), F(5x5,3x3), F(6x6,3x3) and (three-stage) "
                "F(7x7,3x3) are supported", m);
        return WINO_EINVAL;
    }
    const long long T = m + 2, TH = (H + m - 1) / m, TW = (W + m - 1) / m;
    const long long ntiles = (long long)N * TH * TW;
    const long long xel = (long long)N * C * H * W, yel = (long long)N * K * H * W;
    const long long lim = (1LL << 31) / 4;  // elements below 2^31 bytes
    if (xel >= lim || yel >= lim || ntiles >= (1LL << 30) || (long long)H * W >= lim) {
        set_err("problem too large: x and y must each stay below 2^31 bytes");
        return WINO_EUNSUPPORTED;
    }
    g->N = N; g->C = C; g->K = K; g->H = H; g->W = W; g->m = m;
    g->T = (int)T;
    g->T2 = algo == WINO_ALGO_FFT ? (int)(T * (T / 2 + 1)) : (int)(T * T);
    g->TH = (int)TH;
    g->TW = (int)TW;
    g->ntiles = (int)ntiles;
    g->Cs = (C + 3) / 4;
    g->Kb = (K + 15) / 16;
    g->Kb_alloc = (g->Kb + 3) / 4 * 4;
    g->tiles_p = (int)((ntiles + 63) / 64 * 64);
    return WINO_OK;
}

namespace {

bool fail_alloc_forced() {
    const char *e = getenv("WINO_TEST_FAIL_ALLOC");
    return e && e[0] == '1';
}

}  // namespace

// Checks that p (bytes long) is a device allocation on `device` that holds it.
int wino::check_device_ptr(const void *p, size_t bytes, int device, const char *name) {
    if (!p) {
        set_err("%s is NULL", name);
        return WINO_EINVAL;
    }
    if ((reinterpret_cast<uintptr_t>(p) & 3u) != 0) {
        set_err("%s is not 4-byte aligned", name);
        return WINO_EINVAL;
    }
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof attr);
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        set_err("%s is not a HIP device allocation (%s)", name, hipGetErrorString(e));
        return WINO_EINVAL;
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) {
        set_err("%s is not device memory", name);
        return WINO_EINVAL;
    }
    if (attr.device != device) {
        set_err("%s is on device %d, the plan on device %d", name, attr.device, device);
        return WINO_EINVAL;
    }
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    e = hipMemGetAddressRange(&base, &size, const_cast<void *>(p));
    if (e == hipSuccess && base) {
        const uintptr_t b = reinterpret_cast<uintptr_t>(base), q = reinterpret_cast<uintptr_t>(p);
        if (q + bytes > b + size) {
            set_err("%s: the allocation holds %zu bytes from this pointer, the tensor needs %zu",
                    name, (size_t)(b + size - q), bytes);
            return WINO_EINVAL;
        }
    } else {
        (void)hipGetLastError();
    }
    return WINO_OK;
}

bool wino::overlap(const void *a, size_t na, const void *b, size_t nb) {
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + nb && y < x + na;
}

int wino::check_stream_device(hipStream_t s, int device) {
    if (!s) return WINO_OK;  // null stream of the current device
    hipDevice_t dev = -1;
    hipError_t e = hipStreamGetDevice(s, &dev);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        set_err("invalid stream (%s)", hipGetErrorString(e));
        return WINO_EINVAL;
    }
    if (dev != device) {
        set_err("stream is on device %d, the plan on device %d", dev, device);
        return WINO_EINVAL;
    }
    return WINO_OK;
}

namespace {

using wino::check_device_ptr;
using wino::make_geometry;
using wino::overlap;

int check_stream(const wino_plan *p, hipStream_t s) { return wino::check_stream_device(s, p->device); }

size_t x_bytes(const Geometry &g) { return (size_t)g.N * g.C * g.H * g.W * 4; }
size_t y_bytes(const Geometry &g) { return (size_t)g.N * g.K * g.H * g.W * 4; }
size_t w_bytes(const Geometry &g) { return (size_t)g.K * g.C * 9 * 4; }

// Runs the transformed-domain part (everything after the kernel transform).
int run_body(const wino_plan *p, const float *x, float *y, hipStream_t s) {
    hipError_t e;
    if (p->algo == WINO_ALGO_FUSED) {
        e = wino::launch_fused(p->g, p->fcfg, x, p->wt, y, p->split, s);
        if (e != hipSuccess) return hip_fail("fused kernel launch", e);
    } else if (p->algo == WINO_ALGO_FFT) {
        e = wino::launch_fft_fused(p->g, x, p->wt, y, s);
        if (e != hipSuccess) return hip_fail("FFT kernel launch", e);
    } else {
        e = wino::launch_input_transform(p->g, x, p->U, s);
        if (e != hipSuccess) return hip_fail("input transform launch", e);
        e = wino::launch_frequency_gemm(p->g, p->U, p->wt, p->Mf, s);
        if (e != hipSuccess) return hip_fail("frequency product launch", e);
        e = wino::launch_output_transform(p->g, p->Mf, y, s);
        if (e != hipSuccess) return hip_fail("output transform launch", e);
    }
    return WINO_OK;
}

int check_io(const wino_plan *p, const float *x, float *y, hipStream_t s) {
    int rc;
    if ((rc = check_stream(p, s)) != WINO_OK) return rc;
    if ((rc = check_device_ptr(x, x_bytes(p->g), p->device, "x")) != WINO_OK) return rc;
    if ((rc = check_device_ptr(y, y_bytes(p->g), p->device, "y")) != WINO_OK) return rc;
    if (overlap(x, x_bytes(p->g), y, y_bytes(p->g))) {
        set_err("y overlaps x");
        return WINO_EINVAL;
    }
    return WINO_OK;
}

}  // namespace

// Error reporting for the other translation units of the library.
void wino::set_error(const char *fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_err = buf;
}

extern "C" {

const char *wino_last_error(void) { return g_err.c_str(); }

wino_plan *wino_conv_plan_ex(int N, int C, int K, int H, int W, int m, int algo,
                             const wino_tuning *t) {
    Geometry g;
    if (algo != WINO_ALGO_FUSED && algo != WINO_ALGO_THREE_STAGE && algo != WINO_ALGO_FFT) {
        set_err("unknown algorithm %d", algo);
        return nullptr;
    }
    if (make_geometry(N, C, K, H, W, m, algo, &g) != WINO_OK) return nullptr;
    // blocking overrides (checked here, before any HIP call)
    int want_R = 0, want_kit = 0, csplit = 0;
    if (t) {
        if (t->tiles_per_wg < 0 || t->k_per_wg < 0 || t->c_chunk < 0 || t->channel_splits < 0) {
            set_err("tuning fields must be >= 0");
            return nullptr;
        }
        if ((t->tiles_per_wg || t->k_per_wg || t->c_chunk || t->channel_splits > 1) && algo != WINO_ALGO_FUSED) {
            set_err("blocking overrides apply to the fused algorithm only");
            return nullptr;
        }
        want_R = t->tiles_per_wg;
        want_kit = t->k_per_wg;
        if (t->c_chunk) {
            const int R = want_R ? want_R : (m == 2 ? 32 : 16);
            if (t->c_chunk * R != 256) {
                set_err("c_chunk=%d: a stage holds 256 / tiles_per_wg = %d input channels", t->c_chunk, 256 / R);
                return nullptr;
            }
            want_R = R;
        }
        bool any = false;
        for (const wino::FusedBlocking &b : wino::kFusedBlockings)
            if (b.m == m && (!want_R || b.R == want_R) && (!want_kit || b.kit == want_kit)) any = true;
        if (algo == WINO_ALGO_FUSED && !any) {
            set_err("fused blocking tiles_per_wg=%d k_per_wg=%d is not built for m=%d", want_R, want_kit, m);
            return nullptr;
        }
        if (t->channel_splits > 1) {
            if (t->channel_splits > WINO_MAX_CHANNEL_SPLITS) {
                set_err("channel_splits=%d exceeds %d", t->channel_splits, WINO_MAX_CHANNEL_SPLITS);
                return nullptr;
            }
            csplit = t->channel_splits;
        }
    }
    // frequencies in float4 groups, the last one padded when T^2 is odd (F(5));
    // FFT: a float4 {Re, Im, -Im, 0} per frequency
    const size_t wt_bytes = algo == WINO_ALGO_FFT
                                ? (size_t)g.Cs * 4 * g.Kb * 16 * g.T2 * 4 * sizeof(float)
                                : (size_t)g.Kb_alloc * 16 * g.Cs * 4 * ((g.T2 + 3) / 4 * 4) * sizeof(float);
    size_t U_bytes = 0, M_bytes = 0;
    if (algo == WINO_ALGO_THREE_STAGE) {
        // frequencies padded to whole float4s (F(5): 49 -> 52)
        const size_t T2p = (size_t)(g.T2 + 3) / 4 * 4;
        U_bytes = T2p * g.Cs * 4 * g.tiles_p * sizeof(float);
        M_bytes = T2p * g.Kb_alloc * 16 * g.tiles_p * sizeof(float);
    }
    // The kernels address the transformed kernels, the input and the output with
    // 32-bit byte offsets (buffer resources): each must stay below 2^32 bytes.
    if (wt_bytes >= (size_t(1) << 32)) {
        set_err("problem too large: the transformed kernels take %zu bytes, the kernels address "
                "at most 2^32 (C=%d K=%d m=%d)", wt_bytes, C, K, m);
        return nullptr;
    }
    if (fail_alloc_forced()) {
        set_err("device allocation of %zu bytes failed (forced by WINO_TEST_FAIL_ALLOC)",
                wt_bytes + U_bytes + M_bytes);
        return nullptr;
    }
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        hip_fail("hipGetDevice", e);
        return nullptr;
    }
    int num_cus = 256;
    {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus < 1) {
            (void)hipGetLastError();
            cus = 256;
        }
        num_cus = cus;
    }
    FusedCfg cfg{0, 0, num_cus, csplit};
    if (algo == WINO_ALGO_FUSED) {
        cfg = wino::fused_cfg_default(g, num_cus, want_R, want_kit);
        cfg.csplit = csplit;
    }
    size_t part_bytes = 0, cnt_bytes = 0;
    if (algo == WINO_ALGO_FUSED) {
        const wino::SplitInfo si = wino::fused_split_info(g, cfg);
        if (si.n_tail > 0) {
            part_bytes = (size_t)si.n_tail * si.maxc * si.part_floats * sizeof(float);
            cnt_bytes = (size_t)si.n_tail * sizeof(unsigned);
        }
    }
    // status word (wino_conv_status), 256 bytes so the allocation is its own cache line
    const size_t err_bytes = 256;
    const size_t total_bytes = wt_bytes + U_bytes + M_bytes + part_bytes + cnt_bytes + err_bytes;
    wino_plan *p = new (std::nothrow) wino_plan();
    if (!p) {
        set_err("host allocation failed");
        return nullptr;
    }
    p->g = g;
    p->algo = algo;
    p->fcfg = cfg;
    p->device = dev;
    p->wt_bytes = wt_bytes;
    p->U_bytes = U_bytes;
    p->M_bytes = M_bytes;
    p->part_bytes = part_bytes;
    p->cnt_bytes = cnt_bytes;
    void *ptr = nullptr;
    if ((e = hipMalloc(&ptr, wt_bytes)) != hipSuccess) goto oom;
    p->wt = static_cast<float *>(ptr);
    if (U_bytes) {
        if ((e = hipMalloc(&ptr, U_bytes)) != hipSuccess) goto oom;
        p->U = static_cast<float *>(ptr);
        if ((e = hipMalloc(&ptr, M_bytes)) != hipSuccess) goto oom;
        p->Mf = static_cast<float *>(ptr);
    }
    if ((e = hipMalloc(&ptr, err_bytes)) != hipSuccess) goto oom;
    p->split.err = static_cast<unsigned *>(ptr);
    if ((e = hipMemset(p->split.err, 0, err_bytes)) != hipSuccess) goto oom;
    if (part_bytes) {
        if ((e = hipMalloc(&ptr, part_bytes)) != hipSuccess) goto oom;
        p->split.part = static_cast<float *>(ptr);
        if ((e = hipMalloc(&ptr, cnt_bytes)) != hipSuccess) goto oom;
        p->split.cnt = static_cast<unsigned *>(ptr);
        // arrival counters start at zero; each split item's last contributor
        // resets its counter, so they are zero again after every call
        if ((e = hipMemset(p->split.cnt, 0, cnt_bytes)) != hipSuccess) goto oom;
    }
    if ((e = hipDeviceSynchronize()) != hipSuccess) goto oom;
    if (log_enabled())
        fprintf(stderr,
                "[wino] plan N=%d C=%d K=%d H=%d W=%d m=%d algo=%s tiles=%d R=%d k_per_wg=%d "
                "channel_splits=%d workspace=%zu B\n",
                N, C, K, H, W, m,
                algo == WINO_ALGO_FUSED ? "fused" : algo == WINO_ALGO_FFT ? "fft" : "three_stage", g.ntiles,
                cfg.R, cfg.kit, cfg.csplit, total_bytes);
    return p;
oom:
    (void)hipGetLastError();
    set_err("device allocation failed (%s); workspace needs %zu bytes", hipGetErrorString(e),
            total_bytes);
    wino_conv_destroy(p);
    return nullptr;
}

int wino_conv_plan_params(const wino_plan *p, int *m, int *algo, int *tiles_per_wg, int *k_per_wg) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    if (m) *m = p->g.m;
    if (algo) *algo = p->algo;
    if (tiles_per_wg) *tiles_per_wg = p->algo == WINO_ALGO_FUSED ? p->fcfg.R : 0;
    if (k_per_wg) *k_per_wg = p->algo == WINO_ALGO_FUSED ? p->fcfg.kit : 0;
    return WINO_OK;
}

int wino_fused_blockings(int *m, int *tiles_per_wg, int *k_per_wg, int max) {
    int n = 0;
    for (const wino::FusedBlocking &b : wino::kFusedBlockings) {
        if (n < max) {
            if (m) m[n] = b.m;
            if (tiles_per_wg) tiles_per_wg[n] = b.R;
            if (k_per_wg) k_per_wg[n] = b.kit;
        }
        ++n;
    }
    return n;
}

wino_plan *wino_conv_plan(int N, int C, int K, int H, int W, int m) {
    return wino_conv_plan_ex(N, C, K, H, W, m, WINO_ALGO_FUSED, nullptr);
}

void wino_conv_destroy(wino_plan *p) {
    if (!p) return;
    if (p->wt) (void)hipFree(p->wt);
    if (p->U) (void)hipFree(p->U);
    if (p->Mf) (void)hipFree(p->Mf);
    if (p->split.part) (void)hipFree(p->split.part);
    if (p->split.cnt) (void)hipFree(p->split.cnt);
    if (p->split.err) (void)hipFree(p->split.err);
    delete p;
}

size_t wino_conv_workspace_bytes(const wino_plan *p) {
    return p ? p->wt_bytes + p->U_bytes + p->M_bytes + p->part_bytes + p->cnt_bytes + 256 : 0;
}

int wino_conv_status(const wino_plan *p) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail("hipDeviceSynchronize", e);
    unsigned word = 0;
    e = hipMemcpy(&word, p->split.err, sizeof word, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail("hipMemcpy of the status word", e);
    if (word == 0) return WINO_OK;
    // clear the word, and the split arrival counters a wait that gave up may have
    // left nonzero, so that the next call starts clean
    e = hipMemset(p->split.err, 0, sizeof word);
    if (e == hipSuccess && p->split.cnt) e = hipMemset(p->split.cnt, 0, p->cnt_bytes);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail("resetting the status word", e);
    set_err("a kernel wait gave up (status 0x%x): the outputs of the calls since the last "
            "status check are not valid", word);
    return WINO_EKERNEL;
}

int wino_conv_describe(const wino_plan *p, char *buf, size_t len) {
    if (!p || !buf || len == 0) {
        set_err("plan or buffer is NULL, or len is 0");
        return WINO_EINVAL;
    }
    if (p->algo == WINO_ALGO_FUSED) {
        wino::describe_fused(p->g, p->fcfg, buf, len);
    } else if (p->algo == WINO_ALGO_FFT) {
        snprintf(buf, len, "fft_weight_transform_kernel, fft_fused_kernel: 16 x 16 tiles, 16 tiles x 16 output "
                 "channels per work item");
    } else {
        wino::describe_three_stage(p->g, buf, len);
    }
    return WINO_OK;
}

int wino_conv_debug_set_status(const wino_plan *p, unsigned word) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    hipError_t e = hipMemcpy(p->split.err, &word, sizeof word, hipMemcpyHostToDevice);
    if (e != hipSuccess) return hip_fail("hipMemcpy of the status word", e);
    return WINO_OK;
}

int wino_conv_info(const wino_plan *p, long long *n_tiles, double *direct_flops,
                   double *tdomain_flops) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    const Geometry &g = p->g;
    if (n_tiles) *n_tiles = g.ntiles;
    if (direct_flops) *direct_flops = 2.0 * g.N * g.C * g.K * g.H * g.W * 9.0;
    // FFT: T2 complex frequencies, four real multiply-adds per complex one
    const double per = p->algo == WINO_ALGO_FFT ? 8.0 * g.T2 : 2.0 * g.T2;
    if (tdomain_flops) *tdomain_flops = per * (double)g.ntiles * g.C * g.K;
    return WINO_OK;
}

int wino_conv_run(const wino_plan *p, const float *x, const float *w, float *y, void *stream) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int rc;
    if ((rc = check_io(p, x, y, s)) != WINO_OK) return rc;
    if ((rc = check_device_ptr(w, w_bytes(p->g), p->device, "w")) != WINO_OK) return rc;
    if (overlap(w, w_bytes(p->g), y, y_bytes(p->g))) {
        set_err("y overlaps w");
        return WINO_EINVAL;
    }
    hipError_t e = p->algo == WINO_ALGO_FFT ? wino::launch_fft_weight_transform(p->g, w, p->wt, s)
                                            : wino::launch_weight_transform(p->g, w, p->wt, s);
    if (e != hipSuccess) return hip_fail("kernel transform launch", e);
    p->weights_set = true;  // wt now holds this call's kernels
    return run_body(p, x, y, s);
}

int wino_conv_set_weights(wino_plan *p, const float *w, void *stream) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int rc;
    if ((rc = check_stream(p, s)) != WINO_OK) return rc;
    if ((rc = check_device_ptr(w, w_bytes(p->g), p->device, "w")) != WINO_OK) return rc;
    hipError_t e = p->algo == WINO_ALGO_FFT ? wino::launch_fft_weight_transform(p->g, w, p->wt, s)
                                            : wino::launch_weight_transform(p->g, w, p->wt, s);
    if (e != hipSuccess) return hip_fail("kernel transform launch", e);
    p->weights_set = true;
    return WINO_OK;
}

int wino_conv_run_pretransformed(const wino_plan *p, const float *x, float *y, void *stream) {
    if (!p) {
        set_err("plan is NULL");
        return WINO_EINVAL;
    }
    if (!p->weights_set) {
        set_err("no weights set: call wino_conv_set_weights first (wino_conv_run replaces them)");
        return WINO_EINVAL;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    int rc;
    if ((rc = check_io(p, x, y, s)) != WINO_OK) return rc;
    return run_body(p, x, y, s);
}

int wino_conv_intermediate_dims(const wino_plan *p, int which, long long dims[4]) {
    if (!p || !dims) {
        set_err("plan or dims is NULL");
        return WINO_EINVAL;
    }
    const Geometry &g = p->g;
    switch (which) {
        case WINO_BUF_WEIGHTS:
            if (p->algo == WINO_ALGO_FFT) {
                dims[0] = g.Cs; dims[1] = g.Kb; dims[2] = g.T2; dims[3] = 256;
                return WINO_OK;
            }
            dims[0] = g.Kb_alloc; dims[1] = g.Cs; dims[2] = (g.T2 + 3) / 4 * 4; dims[3] = 64;
            return WINO_OK;
        case WINO_BUF_INPUT:
            if (!p->U) break;
            dims[0] = (g.T2 + 3) / 4; dims[1] = g.tiles_p / 16; dims[2] = g.Cs; dims[3] = 256;
            return WINO_OK;
        case WINO_BUF_PRODUCT:
            if (!p->Mf) break;
            dims[0] = (g.T2 + 3) / 4; dims[1] = g.tiles_p / 16; dims[2] = g.Kb_alloc; dims[3] = 1024;
            return WINO_OK;
        default:
            break;
    }
    set_err("plan has no intermediate buffer %d", which);
    return WINO_EINVAL;
}

int wino_conv_copy_intermediate(const wino_plan *p, int which, float *host_dst, size_t count) {
    if (!p || !host_dst) {
        set_err("plan or destination is NULL");
        return WINO_EINVAL;
    }
    const float *src = nullptr;
    size_t bytes = 0;
    switch (which) {
        case WINO_BUF_WEIGHTS: src = p->wt; bytes = p->wt_bytes; break;
        case WINO_BUF_INPUT: src = p->U; bytes = p->U_bytes; break;
        case WINO_BUF_PRODUCT: src = p->Mf; bytes = p->M_bytes; break;
        default: break;
    }
    if (!src) {
        set_err("plan has no intermediate buffer %d", which);
        return WINO_EINVAL;
    }
    if (count * sizeof(float) > bytes) {
        set_err("asked for %zu floats, the buffer holds %zu", count, bytes / sizeof(float));
        return WINO_EINVAL;
    }
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail("hipDeviceSynchronize", e);
    e = hipMemcpy(host_dst, src, count * sizeof(float), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return hip_fail("hipMemcpy", e);
    return WINO_OK;
}

}  // extern "C"
